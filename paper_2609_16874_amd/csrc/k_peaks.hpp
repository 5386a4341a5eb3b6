// k_peaks.hpp -- local-maxima search and compaction (Section 3.2, "Local
// Maxima Search") by one workgroup.
//
// Sums the replicated vote histograms (and clears them for the next frame),
// marks every bin whose count exceeds the threshold and every in-range
// 8-neighbour, and compacts the marked bins in ascending bin order
// b * B_w + a with wave ballots and a prefix sum over the waves.  Writes the
// centroid records, the true count K, the compact peak list and, for grids up
// to 32 x 32, the candidate batches and the bin -> centroid-index table used
// by the matrix-core assignment kernel.
//
// For grids up to 32 x 32 this runs in the tail of the vote kernel, in the
// last workgroup to finish; larger grids use the stand-alone kernel k_peaks.
//
// Candidate batches.  The first min(K, cap) peaks are grouped by row b into
// batches of 4 columns (a row's last batch repeats its last column, which
// leaves a minimum unchanged).  Batch i is bofs[i] = the byte offsets a * 256
// of its 4 columns in the assignment kernel's [bin][64 pixels] x-key array,
// and bhdr[i] = 128 b, which is both the byte offset of row b in its
// [bin][64 pixels] 16-bit y-code array and the row's bits of the search key.
// The list is padded to a multiple of 4 batches with copies of its last one.
#pragma once

#include "cpe_common.hpp"

namespace cpe {

struct PeakOut {
    cpe_centroid *cents;          // caller's centroid records [cap]
    int32_t *num;                 // caller's K
    int32_t *peaks;               // [cap] a | b << 16
    int32_t *kinfo;               // [0] = min(K, cap), [1] = K, [2] = candidate batches
    uint32_t *bofs;               // [kMaxBatch][4] candidate batch column offsets
    uint32_t *bhdr;               // [kMaxBatch] candidate batch row words
    uint16_t *rank;               // [32 * 32] centroid index of peak bin (a, b) at b * 32 + a
};

// Block-level scratch of peak_extract (static LDS).
struct PeakScratch {
    int wave[16];
    int base;
    uint32_t rowmask[kMfmaBins];  // bit a of row b: (a, b) is one of the first min(K, cap) peaks
    int nbt[kMfmaBins];
};

// The whole extraction; every thread of the block calls it.  s_h: LDS
// scratch of Bw * Bh u64.  The replicas are read with device-scope atomic
// loads, so this is also correct in the workgroup that finishes the vote
// kernel (after its acquire fence).  KU bins per thread are summed at a time
// (KU x kReplicas loads in flight).
template <int KU>
__device__ __forceinline__ void peak_extract(unsigned long long *__restrict__ hrep,
                                             unsigned long long *__restrict__ hlast, int32_t Bw, int32_t Bh,
                                             long long cut, int32_t cap, const float *__restrict__ cx,
                                             const float *__restrict__ cy, const PeakOut &po,
                                             unsigned long long *s_h, PeakScratch &ps)
{
    const int tid = threadIdx.x;
    const int nb = Bw * Bh;
    // KU bins per thread and pass, all their loads issued before any is used
    // (out-of-range bins read bin 0 and are discarded)
    constexpr int kU = KU;
    for (int i0 = 0; i0 < nb; i0 += kU * (int)blockDim.x) {
        int idx[kU];
#pragma unroll
        for (int u = 0; u < kU; u++) {
            const int i = i0 + u * (int)blockDim.x + tid;
            idx[u] = i < nb ? i : 0;
        }
        unsigned long long v[kReplicas][kU];
#pragma unroll
        for (int r = 0; r < kReplicas; r++)
#pragma unroll
            for (int u = 0; u < kU; u++)
                v[r][u] = __hip_atomic_load(hrep + (size_t)r * nb + idx[u], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int u = 0; u < kU; u++) {
            unsigned long long s = 0;
#pragma unroll
            for (int r = 0; r < kReplicas; r++) s += v[r][u];
            const int i = i0 + u * (int)blockDim.x + tid;
            if (i < nb) {
#pragma unroll
                for (int r = 0; r < kReplicas; r++) hrep[(size_t)r * nb + i] = 0ull;
                s_h[i] = s;
                hlast[i] = s;
            }
        }
    }
    if (tid == 0) ps.base = 0;
    if (tid < kMfmaBins) ps.rowmask[tid] = 0u;
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
        if (lane == 0) ps.wave[wid] = __popcll(mask);
        __syncthreads();
        int off = ps.base;
        for (int w = 0; w < wid; w++) off += ps.wave[w];
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
                    atomicOr(&ps.rowmask[b], 1u << a);
                    po.rank[b * kMfmaBins + a] = (uint16_t)pos;
                }
            }
        }
        __syncthreads();
        if (tid == 0) {
            int tot = 0;
            for (int w = 0; w < nwaves; w++) tot += ps.wave[w];
            ps.base += tot;
        }
        __syncthreads();
    }
    if (small) {                  // uniform: every thread takes the same branch
        // strict maxima are never horizontally adjacent: <= 16 per row, <= 4 batches
        if (tid < kMfmaBins) ps.nbt[tid] = min((__popc(ps.rowmask[tid]) + 3) >> 2, kMaxBatch / kMfmaBins);
        __syncthreads();
        if (tid < kMfmaBins) {
            const int b = tid;
            int start = 0, total = 0;
            for (int r = 0; r < kMfmaBins; r++) {
                const int n = ps.nbt[r];
                start += r < b ? n : 0;
                total += n;
            }
            uint32_t m = ps.rowmask[b], last = 0;
            const int nbt = ps.nbt[b];
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
            // pad the list to a multiple of 4 with copies of the last batch (a
            // repeated batch leaves every minimum unchanged)
            const int padded = (total + 3) & ~3;
            if (nbt > 0 && start + nbt == total) {
                for (int e = total; e < padded; e++) {
                    for (int s = 0; s < 4; s++) po.bofs[(size_t)e * 4 + s] = po.bofs[(size_t)(total - 1) * 4 + s];
                    po.bhdr[e] = po.bhdr[total - 1];
                }
            }
            if (b == 0) po.kinfo[2] = padded;
        }
    }
    if (tid == 0) {
        *po.num = ps.base;
        po.kinfo[0] = ps.base < cap ? ps.base : cap;
        po.kinfo[1] = ps.base;
    }
}

namespace {   // one private copy per translation unit that launches it

__global__ __launch_bounds__(1024) void k_peaks(unsigned long long *__restrict__ hrep,
                                                unsigned long long *__restrict__ hlast, int32_t Bw, int32_t Bh,
                                                long long cut, int32_t cap, const float *__restrict__ cx,
                                                const float *__restrict__ cy, PeakOut po)
{
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ PeakScratch ps;
    peak_extract<1>(hrep, hlast, Bw, Bh, cut, cap, cx, cy, po, reinterpret_cast<unsigned long long *>(smem), ps);
}

}  // namespace

}  // namespace cpe
