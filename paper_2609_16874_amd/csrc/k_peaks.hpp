// k_peaks.hpp -- local-maxima search and compaction (Section 3.2, "Local
// Maxima Search"), one workgroup of 1024 threads per frame.
//
// Sums the replicated vote histograms (and clears them for the next frame),
// marks every bin whose count exceeds the threshold and every in-range
// 8-neighbour, and compacts the marked bins in ascending bin order
// b * B_w + a with wave ballots and a prefix sum over the waves.  Writes the
// centroid records, the true count K, the compact peak list and, for grids up
// to 32 x 32, the candidate batches and the bin -> centroid-index table used
// by the matrix-core assignment kernel.
//
// Candidate batches.  The first min(K, cap) peaks are grouped by row b into
// batches of 4 columns (a row's last batch repeats its last column, which
// leaves a minimum unchanged).  Batch i is bofs[i] = the byte offsets a * 256
// of its 4 columns in the assignment kernel's [bin][64 pixels] x-key array,
// and bhdr[i] = 128 b, which is both the byte offset of row b in its
// [bin][64 pixels] 16-bit y-code array and the row's bits of the search key.
// Entry nbat (one past the last) is zero, so a one-ahead prefetch stays
// inside the list.
#pragma once

#include "cpe_common.hpp"

namespace cpe {

struct PeakOut {
    cpe_centroid *cents;          // caller's centroid records [cap]
    int32_t *num;                 // caller's K
    int32_t *peaks;               // [cap] a | b << 16
    int32_t *kinfo;               // [0] = min(K, cap), [1] = K
    uint32_t *bofs;               // [kMaxBatch + 1][4] candidate batch column offsets
    uint32_t *bhdr;               // [kMaxBatch + 1] candidate batch row words
    uint16_t *rank;               // [32 * 32] centroid index of peak bin (a, b) at b * 32 + a
};

namespace {   // one private copy per translation unit that launches it

__global__ __launch_bounds__(1024) void k_peaks(unsigned long long *__restrict__ hrep,
                                                unsigned long long *__restrict__ hlast, int32_t Bw, int32_t Bh,
                                                long long cut, int32_t cap, const float *__restrict__ cx,
                                                const float *__restrict__ cy, PeakOut po)
{
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned long long *s_h = reinterpret_cast<unsigned long long *>(smem);   // [nb]
    __shared__ int s_wave[16];
    __shared__ int s_base;
    __shared__ uint32_t s_rowmask[kMfmaBins];   // bit a of row b: (a, b) is one of the first min(K, cap) peaks
    __shared__ int s_nbt[kMfmaBins];
    const int tid = threadIdx.x;
    const int nb = Bw * Bh;
    for (int i = tid; i < nb; i += blockDim.x) {
        unsigned long long s = 0;
#pragma unroll
        for (int r = 0; r < kReplicas; r++) s += hrep[(size_t)r * nb + i];
#pragma unroll
        for (int r = 0; r < kReplicas; r++) hrep[(size_t)r * nb + i] = 0ull;
        s_h[i] = s;
        hlast[i] = s;
    }
    if (tid == 0) s_base = 0;
    if (tid < kMfmaBins) s_rowmask[tid] = 0u;
    __syncthreads();

    const bool small = Bw <= kMfmaBins && Bh <= kMfmaBins;
    const int lane = tid & 63, wid = tid >> 6, nwaves = blockDim.x >> 6;
    for (int c0 = 0; c0 < nb; c0 += blockDim.x) {
        const int i = c0 + tid;
        bool flag = false;
        int a = 0, b = 0;
        unsigned long long v = 0;
        if (i < nb) {
            a = i % Bw;
            b = i / Bw;
            v = s_h[i];
            flag = (long long)v > cut;
            for (int db = -1; db <= 1; db++)
                for (int da = -1; da <= 1; da++) {
                    if (!da && !db) continue;
                    const int nb_ = b + db, na = a + da;
                    if (nb_ < 0 || nb_ >= Bh || na < 0 || na >= Bw) continue;
                    if (!(v > s_h[nb_ * Bw + na])) flag = false;
                }
        }
        const unsigned long long mask = __ballot(flag);
        const int before = lane_prefix(mask);
        if (lane == 0) s_wave[wid] = __popcll(mask);
        __syncthreads();
        int off = s_base;
        for (int w = 0; w < wid; w++) off += s_wave[w];
        if (flag) {
            const int pos = off + before;
            if (pos < cap) {
                cpe_centroid rec;
                rec.bin_x = a;
                rec.bin_y = b;
                rec.x = cx[a];
                rec.y = cy[b];
                rec.score = (double)v * 0x1p-30;
                rec.npix = 0;
                rec.reserved = 0;
                po.cents[pos] = rec;
                po.peaks[pos] = a | (b << 16);
                if (small) {
                    atomicOr(&s_rowmask[b], 1u << a);
                    po.rank[b * kMfmaBins + a] = (uint16_t)pos;
                }
            }
        }
        __syncthreads();
        if (tid == 0) {
            int tot = 0;
            for (int w = 0; w < nwaves; w++) tot += s_wave[w];
            s_base += tot;
        }
        __syncthreads();
    }
    if (small) {                  // uniform: every thread takes the same branch
        // strict maxima are never horizontally adjacent: <= 16 per row, <= 4 batches
        if (tid < kMfmaBins) s_nbt[tid] = min((__popc(s_rowmask[tid]) + 3) >> 2, kMaxBatch / kMfmaBins);
        __syncthreads();
        if (tid < kMfmaBins) {
            const int b = tid;
            int start = 0, total = 0;
            for (int r = 0; r < kMfmaBins; r++) {
                const int n = s_nbt[r];
                start += r < b ? n : 0;
                total += n;
            }
            uint32_t m = s_rowmask[b], last = 0;
            const int nbt = s_nbt[b];
            for (int j = 0; j < nbt; j++) {
                uint32_t o[4];
                for (int s = 0; s < 4; s++) {
                    if (m) {
                        last = (uint32_t)__builtin_ctz(m) * 256u;
                        m &= m - 1u;
                    }
                    o[s] = last;
                }
                uint32_t *bo = po.bofs + (size_t)(start + j) * 4;
                bo[0] = o[0];
                bo[1] = o[1];
                bo[2] = o[2];
                bo[3] = o[3];
                po.bhdr[start + j] = (uint32_t)b * 128u;
            }
            if (b == 0) {
                for (int s = 0; s < 4; s++) po.bofs[(size_t)total * 4 + s] = 0u;
                po.bhdr[total] = 0u;
                po.kinfo[2] = total;
            }
        }
    }
    if (tid == 0) {
        *po.num = s_base;
        po.kinfo[0] = s_base < cap ? s_base : cap;
        po.kinfo[1] = s_base;
    }
}

}  // namespace

}  // namespace cpe
