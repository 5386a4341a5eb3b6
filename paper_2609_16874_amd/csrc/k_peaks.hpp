// k_peaks.hpp -- local-maxima search and compaction (Section 3.2, "Local
// Maxima Search").
//
// A bin is a candidate centroid when its vote count exceeds the threshold and
// every in-range 8-neighbour; candidates are numbered in ascending bin order
// b * B_w + a (wave ballots and a prefix sum over the waves).  Two forms:
//
//   peaks_lds     grids up to 32 x 32: run by every workgroup of the
//                 matrix-core assignment kernel in its prologue, entirely in
//                 LDS.  Besides the compact list it builds the bin -> index
//                 table and the candidate batches of the assignment search.
//   peak_extract  any grid: the stand-alone kernel k_peaks between the
//                 generic vote and assignment kernels; it writes the records,
//                 K, the compact list and the summed histogram to memory.
//
// Candidate batches.  The first min(K, cap) candidates are grouped by row b
// into batches of 4 columns (a row's last batch repeats its last column,
// which leaves a minimum unchanged).  Batch i is bo[i] = the byte offsets
// a * 128 of its 4 columns in the assignment kernel's [bin][32 pixels] x-key
// array, and bh[i] = 128 b, which is both the byte offset of row b in its
// [bin][32 pixels] y-key array and the row's bits of the search key.  The
// list is padded to a multiple of 8 batches with copies of its last one.
#pragma once

#include "cpe_common.hpp"

namespace cpe {

typedef uint32_t u32x4_pk __attribute__((ext_vector_type(4)));

// Strict local maxima of a B_w x B_h grid are pairwise non-adjacent, so there
// are at most ceil(B_w / 2) * ceil(B_h / 2) of them.
__host__ __device__ constexpr int max_peaks(int Bw, int Bh) { return ((Bw + 1) / 2) * ((Bh + 1) / 2); }

// Strict 8-neighbour local maximum of s_h (LDS, row-major [Bh][Bw]) above
// `cut`; out-of-range neighbours are ignored.
__device__ __forceinline__ bool is_peak(const unsigned long long *s_h, int i, int Bw, int Bh, long long cut)
{
    const int a = i % Bw, b = i / Bw;
    const unsigned long long v = s_h[i];
    bool f = (long long)v > cut;
#pragma unroll
    for (int db = -1; db <= 1; db++)
#pragma unroll
        for (int da = -1; da <= 1; da++) {
            if (!da && !db) continue;
            const int nb_ = b + db, na = a + da;
            const bool in = nb_ >= 0 && nb_ < Bh && na >= 0 && na < Bw;
            const unsigned long long w = s_h[in ? nb_ * Bw + na : i];   // self when out of range
            f = f && (!in || v > w);
        }
    return f;
}

// Block-level scratch of the compaction (LDS).
struct CompactScratch {
    int wave[32];                 // per-wave counts of the two bins per thread
    int base;
};

// Mark and compact the candidates of s_h in ascending bin order into s_pk;
// returns K (every thread).  Two bins per thread and pass, bins
// c0 + u * blockDim + tid.  on_peak(i, pos) runs for every candidate bin i
// at list position pos.
template <typename OnPeak>
__device__ __forceinline__ int compact_peaks(const unsigned long long *s_h, int Bw, int Bh, long long cut, int *s_pk,
                                             CompactScratch &cs, OnPeak on_peak)
{
    const int tid = threadIdx.x, nb = Bw * Bh;
    const int lane = tid & 63, wid = tid >> 6, nwaves = blockDim.x >> 6;
    if (tid == 0) cs.base = 0;
    __syncthreads();
    for (int c0 = 0; c0 < nb; c0 += 2 * (int)blockDim.x) {
        bool flag[2];
        unsigned long long mask[2];
#pragma unroll
        for (int u = 0; u < 2; u++) {
            const int i = c0 + u * (int)blockDim.x + tid;
            flag[u] = i < nb && is_peak(s_h, i, Bw, Bh, cut);
            mask[u] = __ballot(flag[u]);
        }
        if (lane == 0) {
            cs.wave[wid] = __popcll(mask[0]);
            cs.wave[nwaves + wid] = __popcll(mask[1]);
        }
        __syncthreads();
        // all counts of this pass: pass 0 of every wave, then pass 1
        int off0 = cs.base, off1 = cs.base, tot = 0;
#pragma unroll
        for (int w = 0; w < 16; w++) {          // nwaves <= 16; all reads independent
            const int n0 = w < nwaves ? cs.wave[w] : 0, n1 = w < nwaves ? cs.wave[nwaves + w] : 0;
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
                on_peak(i, pos);
            }
        }
        __syncthreads();
        if (tid == 0) cs.base += tot;
        __syncthreads();
    }
    return cs.base;
}

// ---------------------------------------------------------------------------
// Grids up to 32 x 32: candidates in LDS, in the assignment kernel's prologue
// ---------------------------------------------------------------------------
// The histogram is held in a 32 x 32 slot layout, slot b * 32 + a, whose
// order agrees with the bin order b * B_w + a.  The first kPeakThreads
// threads of the block own two slots each: t and t + kPeakThreads.
constexpr int kLdsPeakBins = 32;
constexpr int kPeakThreads = 512;
constexpr int kMaxBatchLds = 128;   // <= 16 strict maxima per row of 32 -> <= 4 batches per row
constexpr int kBatchPad = 8;        // the batch list is padded to a multiple of this
constexpr int kKeyStride = 32;      // words per bin row of the assignment kernel's key arrays

// LDS of peaks_lds (the summed histogram may alias any scratch the caller
// does not need until the peaks are known).
struct PeakLds {
    int wave[2 * kPeakThreads / 64];  // per-wave counts of the two slot passes (slot-owning waves)
    uint32_t rowmask[kLdsPeakBins];   // bit a of row b: (a, b) is one of the first min(K, cap) candidates
    uint32_t colmask;                 // bit a: column a holds one of them
    int K, Kc, nbat;                  // nbat: batches, padded to a multiple of kBatchPad
    int nbat_real;                    // batches before the padding
    int ncol, nrow;                   // candidate columns and rows
    uint8_t colbin[kLdsPeakBins];     // column of column slot j (ascending; 0 past ncol)
    uint8_t rowbin[kLdsPeakBins];     // row of row slot j (ascending; 0 past nrow)
    int pk[max_peaks(kLdsPeakBins, kLdsPeakBins)];   // candidate slots b * 32 + a, ascending
};

// The vote counts of this thread's two slots, summed over the kReplicas
// histograms `hsrc` ([kReplicas][Bh][Bw], written by the previous launch).
// Issued first, so that their latency overlaps the caller's table staging.
struct PeakLoad {
    unsigned long long v[2][kReplicas];
};
__device__ __forceinline__ void peaks_lds_load(const unsigned long long *__restrict__ hsrc, int Bw, int Bh,
                                               PeakLoad &ld)
{
    const int nb = Bw * Bh;
#pragma unroll
    for (int u = 0; u < 2; u++) {
        const int slot = u * kPeakThreads + (int)threadIdx.x, a = slot & 31, b = slot >> 5;
        const bool in = (int)threadIdx.x < kPeakThreads && a < Bw && b < Bh;
#pragma unroll
        for (int r = 0; r < kReplicas; r++) ld.v[u][r] = in ? hsrc[(size_t)r * nb + b * Bw + a] : 0ull;
    }
}

// Strict 8-neighbour local maximum of slot (a, b) of s_h above `cut`;
// out-of-range neighbours are ignored.
__device__ __forceinline__ bool is_peak32(const unsigned long long *s_h, int a, int b, int Bw, int Bh, long long cut)
{
    const unsigned long long v = s_h[b * 32 + a];
    bool f = a < Bw && b < Bh && (long long)v > cut;
#pragma unroll
    for (int db = -1; db <= 1; db++)
#pragma unroll
        for (int da = -1; da <= 1; da++) {
            if (!da && !db) continue;
            const int nb_ = b + db, na = a + da;
            const bool in = nb_ >= 0 && nb_ < Bh && na >= 0 && na < Bw;
            const unsigned long long w = s_h[in ? nb_ * 32 + na : b * 32 + a];   // self when out of range
            f = f && (!in || v > w);
        }
    return f;
}

// The extraction in two parts, called by every thread of a block of at
// least kPeakThreads threads.  peaks_lds_sum stores the summed histogram
// s_h (32 x 32 slots) from the loaded counts; after a barrier of the
// caller's, peaks_lds_find compacts the candidates in ascending bin order
// (pl.pk) and writes K and min(K, cap), the bin -> candidate-index table
// s_rank [32 * 32], the column and row slots (pl.ncol, pl.nrow, pl.colbin,
// pl.rowbin, and the bin constants by slot s_cbs) and the candidate batches
// s_bo / s_bh in slot offsets (pl.nbat of them, a multiple of kBatchPad).  `mid` runs between its first and second barrier
// (the caller's independent work, e.g. loads whose latency the extraction
// hides).
__device__ __forceinline__ void peaks_lds_sum(const PeakLoad &ld, unsigned long long *s_h, PeakLds &pl)
{
    const int tid = threadIdx.x;
    if (tid < kPeakThreads) {
#pragma unroll
        for (int u = 0; u < 2; u++) {
            unsigned long long sum = 0;
#pragma unroll
            for (int r = 0; r < kReplicas; r++) sum += ld.v[u][r];
            s_h[u * kPeakThreads + tid] = sum;
        }
    }
    if (tid < kLdsPeakBins) pl.rowmask[tid] = 0u;
    if (tid == 0) pl.colmask = 0u;
}
template <typename Mid>
__device__ __forceinline__ void peaks_lds_find(int Bw, int Bh, long long cut, int cap, const unsigned long long *s_h,
                                               PeakLds &pl, u32x4_pk *s_bo, uint32_t *s_bh, uint16_t *s_rank,
                                               const uint32_t *s_cb, uint32_t *s_cbs, Mid mid)
{
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    constexpr int kWaves = kPeakThreads / 64;
    const bool own = tid < kPeakThreads;            // wave-uniform
    bool flag[2];
    unsigned long long mask[2];
#pragma unroll
    for (int u = 0; u < 2; u++) {
        const int slot = u * kPeakThreads + tid;
        flag[u] = own && is_peak32(s_h, slot & 31, slot >> 5, Bw, Bh, cut);
        mask[u] = __ballot(flag[u]);
    }
    if (own && lane == 0) {
        pl.wave[wid] = __popcll(mask[0]);
        pl.wave[kWaves + wid] = __popcll(mask[1]);
    }
    __syncthreads();
    mid();
    int off0 = 0, off1 = 0, K = 0;
#pragma unroll
    for (int w = 0; w < kWaves; w++) {
        const int n0 = pl.wave[w], n1 = pl.wave[kWaves + w];
        off0 += w < wid ? n0 : 0;
        off1 += n0 + (w < wid ? n1 : 0);
        K += n0 + n1;
    }
    const int Kc = K < cap ? K : cap;
#pragma unroll
    for (int u = 0; u < 2; u++) {
        if (flag[u]) {
            const int slot = u * kPeakThreads + tid;
            const int pos = (u ? off1 : off0) + lane_prefix(mask[u]);   // < max_peaks(32, 32)
            pl.pk[pos] = slot;
            if (pos < Kc) {
                s_rank[slot] = (uint16_t)pos;
                atomicOr(&pl.rowmask[slot >> 5], 1u << (slot & 31));
                atomicOr(&pl.colmask, 1u << (slot & 31));
            }
        }
    }
    __syncthreads();
    // Slots: the candidate columns and rows, each numbered in ascending
    // order; the assignment computes distances for slots only, and its
    // arrays, batches and bin constants are indexed by slot.  Lane j of the
    // first wave numbers column j and row j and scatters them (and their
    // bin constants, s_cb [2][32] by bin -> s_cbs [2][32] by slot).
    // Batches: lane b builds row b's (strict maxima are never horizontally
    // adjacent: <= 16 per row, <= 4 batches), as slot byte offsets.
    if (tid < 64) {
        const int b = tid;
        uint32_t m = b < kLdsPeakBins ? pl.rowmask[b] : 0u;
        const uint32_t cm = pl.colmask;
        const unsigned long long rows = __ballot(m != 0u);
        const int rslot = lane_prefix(rows);                         // slot of row b if it holds candidates
        if (b < kLdsPeakBins) {
            pl.colbin[b] = 0;
            pl.rowbin[b] = 0;
        }
        if (b < kLdsPeakBins && ((cm >> b) & 1u)) {
            const int cs = __popc(cm & ((1u << b) - 1u));
            pl.colbin[cs] = (uint8_t)b;
            s_cbs[cs] = s_cb[b];
        }
        if (m) {
            pl.rowbin[rslot] = (uint8_t)b;
            s_cbs[kLdsPeakBins + rslot] = s_cb[kLdsPeakBins + b];
        }
        const int nbt = (__popc(m) + 3) >> 2;
        const int incl = wave_incl_sum(nbt);      // the whole first wave is active here
        const int start = incl - nbt, total = __builtin_amdgcn_readlane(incl, 31);
        const int padded = (total + kBatchPad - 1) & ~(kBatchPad - 1);
        const uint32_t hb = (uint32_t)rslot * (4u * kKeyStride);
        uint32_t last = 0;
        u32x4_pk o = {0u, 0u, 0u, 0u};
        for (int j = 0; j < nbt; j++) {
#pragma unroll
            for (int s4 = 0; s4 < 4; s4++) {
                if (m) {
                    const int a = __builtin_ctz(m);
                    last = (uint32_t)__popc(cm & ((1u << a) - 1u)) * (4u * kKeyStride);
                    m &= m - 1u;
                }
                o[s4] = last;
            }
            s_bo[start + j] = o;
            s_bh[start + j] = hb;
        }
        // pad the list with copies of the last batch (a repeated batch leaves
        // every minimum unchanged)
        if (nbt > 0 && start + nbt == total)
            for (int e = total; e < padded; e++) {
                s_bo[e] = o;
                s_bh[e] = hb;
            }
        if (tid == 0) {
            pl.K = K;
            pl.Kc = Kc;
            pl.nbat = padded;
            pl.nbat_real = total;
            pl.ncol = __popc(cm);
            pl.nrow = __popcll(rows);
        }
    }
    __syncthreads();
}

// ---------------------------------------------------------------------------
// Any grid: the stand-alone peak kernel of the generic path
// ---------------------------------------------------------------------------
struct PeakOut {
    cpe_centroid *cents;          // caller's centroid records [cap]
    int32_t *num;                 // caller's K
    int32_t *peaks;               // [cap] a | b << 16
    int32_t *kinfo;               // [0] = min(K, cap), [1] = K
};

// The whole extraction; every thread of the block calls it.  s_h: LDS
// scratch of Bw * Bh u64; s_pk: LDS scratch of max_peaks(Bw, Bh) ints.
// Until the last barrier every result goes to LDS only, so that no barrier
// waits for global stores; the outputs are written at the end.
__device__ __forceinline__ void peak_extract(const unsigned long long *__restrict__ hrep,
                                             unsigned long long *__restrict__ hlast, int32_t Bw, int32_t Bh,
                                             long long cut, int32_t cap, const float *__restrict__ cx,
                                             const float *__restrict__ cy, const PeakOut &po,
                                             unsigned long long *s_h, int *s_pk, CompactScratch &cs)
{
    const int tid = threadIdx.x;
    const int nb = Bw * Bh;
    for (int i = tid; i < nb; i += blockDim.x) {
        unsigned long long v[kReplicas];
#pragma unroll
        for (int r = 0; r < kReplicas; r++) v[r] = hrep[(size_t)r * nb + i];
        unsigned long long sum = 0;
#pragma unroll
        for (int r = 0; r < kReplicas; r++) sum += v[r];
        s_h[i] = sum;
    }
    const int K = compact_peaks(s_h, Bw, Bh, cut, s_pk, cs, [](int, int) {});
    const int Kc = K < cap ? K : cap;

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
    }
    for (int i = tid; i < nb; i += blockDim.x) hlast[i] = s_h[i];
    if (tid == 0) {
        *po.num = K;
        po.kinfo[0] = Kc;
        po.kinfo[1] = K;
    }
}

namespace {   // one private copy per translation unit that launches it

__global__ __launch_bounds__(1024) void k_peaks(const unsigned long long *__restrict__ hrep,
                                                unsigned long long *__restrict__ hlast, int32_t Bw, int32_t Bh,
                                                long long cut, int32_t cap, const float *__restrict__ cx,
                                                const float *__restrict__ cy, PeakOut po)
{
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ CompactScratch cs;
    unsigned long long *s_h = reinterpret_cast<unsigned long long *>(smem);    // [Bw * Bh]
    int *s_pk = reinterpret_cast<int *>(s_h + Bw * Bh);                          // [max_peaks(Bw, Bh)]
    peak_extract(hrep, hlast, Bw, Bh, cut, cap, cx, cy, po, s_h, s_pk, cs);
}

}  // namespace

}  // namespace cpe
