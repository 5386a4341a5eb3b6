// k_generic.hpp -- decoder kernels for any bin grid up to 128 x 128.
//
// One thread per foreground pixel computes the per-axis squared distances to
// every palette entry with packed 16-bit dot products (Eq4/Eq10), and
//   k_vote_generic    turns them into bucket weights and accumulates the soft
//                     votes (Eq6/Eq11) into a register-tiled 64-bit
//                     histogram, flushed with global atomics into one of the
//                     replicated histograms;
//   k_assign_generic  turns them into distances sqrt_cr(fl32(S)), assigns the
//                     pixel to the candidate with the smallest exact distance
//                     sum (Eq7, lowest index on ties), writes its label and
//                     score and counts it.
// Grids up to 32 x 32 bins use the matrix-core kernels of k_mfma.hpp instead.
#pragma once

#include "cpe_common.hpp"

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
// S1 + S2: recovery and soft voting
// ---------------------------------------------------------------------------
template <typename T, int F>
__global__ __launch_bounds__(256) void k_vote_generic(const T *__restrict__ emb, int32_t dstride, int32_t yoff,
                                              const T *__restrict__ fg, int32_t npix,
                                              float fg_thr, Tables tb, int32_t Bw, int32_t Bh,
                                              unsigned long long *__restrict__ hrep)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int TP = blockDim.x;
    const int tid = threadIdx.x;
    int32_t *s_px = reinterpret_cast<int32_t *>(smem);
    int32_t *s_py = s_px + Bw * F;
    uint32_t *s_nx = reinterpret_cast<uint32_t *>(s_py + Bh * F);
    uint32_t *s_ny = s_nx + Bw;
    int32_t *s_list = reinterpret_cast<int32_t *>(s_ny + Bh);   // [TP]
    int32_t *s_n = s_list + TP;                                  // [4]
    uint16_t *s_wt = reinterpret_cast<uint16_t *>(s_n + 4);      // [kWKeys]
    uint16_t *s_qx = s_wt + kWKeys;                              // [Bw][TP]
    uint16_t *s_qy = s_qx + Bw * TP;                             // [Bh][TP]

    for (int i = tid; i < Bw * F; i += TP) s_px[i] = tb.pal_x[i];
    for (int i = tid; i < Bh * F; i += TP) s_py[i] = tb.pal_y[i];
    for (int i = tid; i < Bw; i += TP) s_nx[i] = tb.n2_x[i];
    for (int i = tid; i < Bh; i += TP) s_ny[i] = tb.n2_y[i];
    for (int i = tid; i < kWKeys; i += TP) s_wt[i] = tb.wt[i];

    using L = PixelLayout<T, F>;
    const int nb = Bw * Bh;
    const int per_chunk = 4 * TP;
    const int nchunks = (nb + per_chunk - 1) / per_chunk;
    unsigned long long *hdst = hrep + (size_t)(blockIdx.x % kReplicas) * nb;

    unsigned long long acc[4] = {0ull, 0ull, 0ull, 0ull};
    int ba[4], bb[4];
#pragma unroll
    for (int j = 0; j < 4; j++) {
        int bin = j * TP + tid;
        ba[j] = bin % Bw;
        bb[j] = (bin / Bw) < Bh ? bin / Bw : 0;
    }

    for (int64_t tile = blockIdx.x; tile * TP < npix; tile += gridDim.x) {
        if (tid == 0) *s_n = 0;
        __syncthreads();
        const int64_t p = tile * TP + tid;
        if (p < npix && fg_value<T>(fg, p) > fg_thr) {
            int slot = atomicAdd(s_n, 1);
            s_list[slot] = (int32_t)p;
        }
        __syncthreads();
        const int n = *s_n;
        if (tid < n) {
            const T *row = emb + (size_t)s_list[tid] * dstride;
            int32_t xk[F], yk[F];
            load_block<T, F, L::kAlignX>(row, xk);
            load_block<T, F, L::kAlignY>(row + yoff, yk);
            const uint32_t nX = (uint32_t)dot_pk<F>(xk, xk);
            const uint32_t nY = (uint32_t)dot_pk<F>(yk, yk);
            for (int a = 0; a < Bw; a++)
                s_qx[a * TP + tid] = s_wt[dist_key<kWMant>(axis_s(nX, s_nx[a], dot_pk<F>(xk, s_px + a * F)))];
            for (int b = 0; b < Bh; b++)
                s_qy[b * TP + tid] = s_wt[dist_key<kWMant>(axis_s(nY, s_ny[b], dot_pk<F>(yk, s_py + b * F)))];
        }
        __syncthreads();
        if (nchunks == 1) {
            for (int i = 0; i < n; i++) {
#pragma unroll
                for (int j = 0; j < 4; j++)
                    acc[j] += (unsigned long long)((uint32_t)s_qx[ba[j] * TP + i] * (uint32_t)s_qy[bb[j] * TP + i]);
            }
        } else {
            for (int c = 0; c < nchunks; c++) {
                unsigned long long part[4] = {0ull, 0ull, 0ull, 0ull};
                int ca[4], cb[4];
#pragma unroll
                for (int j = 0; j < 4; j++) {
                    int bin = c * per_chunk + j * TP + tid;
                    ca[j] = bin % Bw;
                    cb[j] = (bin / Bw) < Bh ? bin / Bw : 0;
                }
                for (int i = 0; i < n; i++) {
#pragma unroll
                    for (int j = 0; j < 4; j++)
                        part[j] += (unsigned long long)((uint32_t)s_qx[ca[j] * TP + i] * (uint32_t)s_qy[cb[j] * TP + i]);
                }
#pragma unroll
                for (int j = 0; j < 4; j++) {
                    int bin = c * per_chunk + j * TP + tid;
                    if (bin < nb && part[j]) atomicAdd(hdst + bin, part[j]);
                }
            }
        }
        __syncthreads();
    }
    if (nchunks == 1) {
#pragma unroll
        for (int j = 0; j < 4; j++) {
            int bin = j * TP + tid;
            if (bin < nb && acc[j]) atomicAdd(hdst + bin, acc[j]);
        }
    }
}

// ---------------------------------------------------------------------------
// S4 + S5: assignment, label write-out, counts
// ---------------------------------------------------------------------------
template <typename T, int F>
__global__ __launch_bounds__(256) void k_assign_generic(const T *__restrict__ emb, int32_t dstride, int32_t yoff,
                                                const T *__restrict__ fg, int32_t npix,
                                                float fg_thr, double tau4096, Tables tb, int32_t Bw, int32_t Bh,
                                                const int32_t *__restrict__ peaks, const int32_t *__restrict__ kinfo,
                                                cpe_centroid *__restrict__ cents, int32_t *__restrict__ labels,
                                                float *__restrict__ score_map)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int TP = blockDim.x;
    const int tid = threadIdx.x;
    int32_t *s_px = reinterpret_cast<int32_t *>(smem);
    int32_t *s_py = s_px + Bw * F;
    uint32_t *s_nx = reinterpret_cast<uint32_t *>(s_py + Bh * F);
    uint32_t *s_ny = s_nx + Bw;
    int32_t *s_list = reinterpret_cast<int32_t *>(s_ny + Bh);   // [TP]
    int32_t *s_n = s_list + TP;                                  // [4]
    int32_t *s_cnt = s_n + 4;                                    // [kCountCap]
    float *s_r = reinterpret_cast<float *>(s_cnt + kCountCap);   // [Bw + Bh][TP] distances

    const int Kc = kinfo[0];
    const int ncnt = Kc < kCountCap ? Kc : kCountCap;
    for (int i = tid; i < Bw * F; i += TP) s_px[i] = tb.pal_x[i];
    for (int i = tid; i < Bh * F; i += TP) s_py[i] = tb.pal_y[i];
    for (int i = tid; i < Bw; i += TP) s_nx[i] = tb.n2_x[i];
    for (int i = tid; i < Bh; i += TP) s_ny[i] = tb.n2_y[i];
    for (int i = tid; i < ncnt; i += TP) s_cnt[i] = 0;

    using L = PixelLayout<T, F>;
    for (int64_t tile = blockIdx.x; tile * TP < npix; tile += gridDim.x) {
        if (tid == 0) *s_n = 0;
        __syncthreads();
        const int64_t p = tile * TP + tid;
        if (p < npix) {
            const bool part = Kc > 0 && fg_value<T>(fg, p) > fg_thr;
            if (part) {
                int slot = atomicAdd(s_n, 1);
                s_list[slot] = (int32_t)p;
            } else {
                labels[p] = 0;
                if (score_map) score_map[p] = 0.0f;
            }
        }
        __syncthreads();
        const int n = *s_n;
        if (tid < n) {
            const int32_t pp = s_list[tid];
            const T *row = emb + (size_t)pp * dstride;
            int32_t xk[F], yk[F];
            load_block<T, F, L::kAlignX>(row, xk);
            load_block<T, F, L::kAlignY>(row + yoff, yk);
            const uint32_t nX = (uint32_t)dot_pk<F>(xk, xk);
            const uint32_t nY = (uint32_t)dot_pk<F>(yk, yk);
            for (int a = 0; a < Bw; a++)
                s_r[a * TP + tid] = sqrt_cr((float)axis_s(nX, s_nx[a], dot_pk<F>(xk, s_px + a * F)));
            for (int b = 0; b < Bh; b++)
                s_r[(Bw + b) * TP + tid] = sqrt_cr((float)axis_s(nY, s_ny[b], dot_pk<F>(yk, s_py + b * F)));
            // Eq7: smallest exact sum (binary64 holds the sum of two binary32
            // values exactly), lowest index on ties
            int best = 0;
            const int32_t pk0 = peaks[0];
            double bd = (double)s_r[(pk0 & 0xffff) * TP + tid] + (double)s_r[(Bw + (pk0 >> 16)) * TP + tid];
            for (int k = 1; k < Kc; k++) {
                const int32_t pk = peaks[k];
                const double d = (double)s_r[(pk & 0xffff) * TP + tid] + (double)s_r[(Bw + (pk >> 16)) * TP + tid];
                if (d < bd) {
                    bd = d;
                    best = k;
                }
            }
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
        __syncthreads();
    }
    __syncthreads();
    for (int i = tid; i < ncnt; i += TP)
        if (s_cnt[i]) atomicAdd(&cents[i].npix, s_cnt[i]);
}


}  // namespace cpe
