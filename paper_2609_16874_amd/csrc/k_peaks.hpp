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

// Block-level scratch of peak_extract (LDS).
struct PeakScratch {
    int wave[32];                 // per-wave counts of the two bins per thread
    int base;
    uint32_t rowmask[kMfmaBins];  // bit a of row b: (a, b) is one of the first min(K, cap) peaks
    int nbt[kMfmaBins];
};

// Strict local maxima of a B_w x B_h grid are pairwise non-adjacent, so there
// are at most ceil(B_w / 2) * ceil(B_h / 2) of them.
__host__ __device__ constexpr int max_peaks(int Bw, int Bh) { return ((Bw + 1) / 2) * ((Bh + 1) / 2); }

// The whole extraction; every thread of the block calls it.  s_h: LDS
// scratch of Bw * Bh u64; s_pk: LDS scratch of max_peaks(Bw, Bh) ints.  The
// replicas are read with device-scope atomic loads, so this is also correct
// in the workgroup that finishes the vote kernel (after its acquire fence).
// KU bins per thread are summed at a time (KU x kReplicas loads in flight).
// Until the last barrier every result goes to LDS only, so that no barrier
// waits for global stores; the outputs are written at the end.
template <int KU>
__device__ __forceinline__ void peak_extract(unsigned long long *__restrict__ hrep,
                                             unsigned long long *__restrict__ hlast, int32_t Bw, int32_t Bh,
                                             long long cut, int32_t cap, const float *__restrict__ cx,
                                             const float *__restrict__ cy, const PeakOut &po,
                                             unsigned long long *s_h, int *s_pk, PeakScratch &ps)
{
    const int tid = threadIdx.x;
    const int nb = Bw * Bh;
    // KU bins per thread and pass, all their loads issued before any is used
    // (out-of-range bins read bin 0 and are discarded)
    for (int i0 = 0; i0 < nb; i0 += KU * (int)blockDim.x) {
        int idx[KU];
#pragma unroll
        for (int u = 0; u < KU; u++) {
            const int i = i0 + u * (int)blockDim.x + tid;
            idx[u] = i < nb ? i : 0;
        }
        unsigned long long v[kReplicas][KU];
#pragma unroll
        for (int r = 0; r < kReplicas; r++)
#pragma unroll
            for (int u = 0; u < KU; u++)
                v[r][u] = __hip_atomic_load(hrep + (size_t)r * nb + idx[u], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int u = 0; u < KU; u++) {
            unsigned long long sum = 0;
#pragma unroll
            for (int r = 0; r < kReplicas; r++) sum += v[r][u];
            const int i = i0 + u * (int)blockDim.x + tid;
            if (i < nb) s_h[i] = sum;
        }
    }
    if (tid == 0) ps.base = 0;
    if (tid < kMfmaBins) ps.rowmask[tid] = 0u;
    __syncthreads();

    // strict local maxima above the threshold, compacted in bin order into
    // s_pk; two bins per thread and pass (bins c0 + u * blockDim + tid)
    const bool small = Bw <= kMfmaBins && Bh <= kMfmaBins;
    const int lane = tid & 63, wid = tid >> 6, nwaves = blockDim.x >> 6;
    for (int c0 = 0; c0 < nb; c0 += 2 * (int)blockDim.x) {
        bool flag[2];
        unsigned long long mask[2];
#pragma unroll
        for (int u = 0; u < 2; u++) {
            const int i = c0 + u * (int)blockDim.x + tid;
            const int ic = i < nb ? i : 0;
            const int a = ic % Bw, b = ic / Bw;
            const unsigned long long v = s_h[ic];
            bool f = i < nb && (long long)v > cut;
#pragma unroll
            for (int db = -1; db <= 1; db++)
#pragma unroll
                for (int da = -1; da <= 1; da++) {
                    if (!da && !db) continue;
                    const int nb_ = b + db, na = a + da;
                    const bool in = nb_ >= 0 && nb_ < Bh && na >= 0 && na < Bw;
                    const unsigned long long w = s_h[in ? nb_ * Bw + na : ic];   // self when out of range
                    f = f && (!in || v > w);
                }
            flag[u] = f;
            mask[u] = __ballot(f);
        }
        if (lane == 0) {
            ps.wave[wid] = __popcll(mask[0]);
            ps.wave[nwaves + wid] = __popcll(mask[1]);
        }
        __syncthreads();
        // all counts of this pass: pass 0 of every wave, then pass 1
        int off0 = ps.base, off1 = ps.base, tot = 0;
#pragma unroll
        for (int w = 0; w < 16; w++) {          // nwaves <= 16; all reads independent
            const int n0 = w < nwaves ? ps.wave[w] : 0, n1 = w < nwaves ? ps.wave[nwaves + w] : 0;
            off0 += w < wid ? n0 : 0;
            off1 += n0 + (w < wid ? n1 : 0);
            tot += n0 + n1;
        }
#pragma unroll
        for (int u = 0; u < 2; u++) {
            if (flag[u]) {
                const int i = c0 + u * (int)blockDim.x + tid;
                const int pos = (u ? off1 : off0) + lane_prefix(mask[u]);   // < max_peaks(Bw, Bh)
                s_pk[pos] = i;
                if (small && pos < cap) atomicOr(&ps.rowmask[i / Bw], 1u << (i % Bw));
            }
        }
        __syncthreads();
        if (tid == 0) ps.base += tot;
        __syncthreads();
    }
    const int K = ps.base, Kc = K < cap ? K : cap;
    if (small) {                  // uniform: every thread takes the same branch
        // strict maxima are never horizontally adjacent: <= 16 per row, <= 4 batches
        if (tid < kMfmaBins) ps.nbt[tid] = min((__popc(ps.rowmask[tid]) + 3) >> 2, kMaxBatch / kMfmaBins);
        __syncthreads();
    }

    // ---- outputs (global stores only from here on) ----
    for (int k = tid; k < Kc; k += blockDim.x) {
        const int i = s_pk[k], a = i % Bw, b = i / Bw;
        cpe_centroid rec;
        rec.bin_x = a;
        rec.bin_y = b;
        rec.x = cx[a];
        rec.y = cy[b];
        rec.score = (double)s_h[i] * 0x1p-30;
        rec.npix = 0;
        rec.reserved = 0;
        po.cents[k] = rec;
        po.peaks[k] = a | (b << 16);
        if (small) po.rank[b * kMfmaBins + a] = (uint16_t)k;
    }
    for (int i = tid; i < nb; i += blockDim.x) {
        hlast[i] = s_h[i];
#pragma unroll
        for (int r = 0; r < kReplicas; r++) hrep[(size_t)r * nb + i] = 0ull;
    }
    if (small && tid < kMfmaBins) {
        const int b = tid;
        int start = 0, total = 0;
        for (int r = 0; r < kMfmaBins; r++) {
            const int n = ps.nbt[r];
            start += r < b ? n : 0;
            total += n;
        }
        uint32_t m = ps.rowmask[b], last = 0;
        const int nbt = ps.nbt[b];
        uint32_t o[4] = {0u, 0u, 0u, 0u};
        for (int j = 0; j < nbt; j++) {
            for (int s4 = 0; s4 < 4; s4++) {
                if (m) {
                    last = (uint32_t)__builtin_ctz(m) * 256u;
                    m &= m - 1u;
                }
                o[s4] = last;
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
                uint32_t *bo = po.bofs + (size_t)e * 4;
                bo[0] = o[0];
                bo[1] = o[1];
                bo[2] = o[2];
                bo[3] = o[3];
                po.bhdr[e] = (uint32_t)b * 128u;
            }
        }
        if (b == 0) po.kinfo[2] = padded;
    }
    if (tid == 0) {
        *po.num = K;
        po.kinfo[0] = Kc;
        po.kinfo[1] = K;
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
    unsigned long long *s_h = reinterpret_cast<unsigned long long *>(smem);    // [Bw * Bh]
    int *s_pk = reinterpret_cast<int *>(s_h + Bw * Bh);                          // [max_peaks(Bw, Bh)]
    peak_extract<1>(hrep, hlast, Bw, Bh, cut, cap, cx, cy, po, s_h, s_pk, ps);
}

}  // namespace

}  // namespace cpe
