// launch.hpp -- the launch sequence of one frame, instantiated per element
// type and harmonic count by the launch_*.hip translation units.
#pragma once

#include <hip/hip_ext.h>

#include "cpe_decoder.hpp"
#include "k_compact.hpp"
#include "k_generic.hpp"
#include "k_mfma.hpp"
#include "k_peaks.hpp"

namespace cpe {

// Grid caps of the matrix-core kernels: one resident vote workgroup (8 or 12
// waves) and one assignment workgroup of 12 waves per compute unit.
constexpr int64_t kVoteGrid = 256;
constexpr int64_t kAssignGrid = 256;
// Frames from this many pixels take the fast assignment search when only
// labels are requested.
constexpr int64_t kFastSearchPixels = 1 << 20;

// Largest pixel tile (threads per block) whose LDS footprint fits the budget.
inline int pick_tile(size_t fixed, size_t per_px, size_t budget)
{
    for (int tp = 256; tp >= 64; tp >>= 1)
        if (fixed + per_px * (size_t)tp <= budget) return tp;
    return 64;
}

template <typename T, int F>
cpe_status launch_all(cpe_decoder *h, const Scratch &sc, const FrameArgs &fa)
{
    hipStream_t stream = fa.stream;
    const float fg_thr = fa.fg_thr;
    const long long cut = fa.cut;
    cpe_centroid *cents = fa.cents;
    int32_t *num = fa.num, *labels = fa.labels;
    float *score = fa.score;
    const void *emb = fa.emb, *fg = fa.fg;
    const int Bw = h->bins_w, Bh = h->bins_h, nb = Bw * Bh;
    const int npix = h->H * h->W;
    const T *e = static_cast<const T *>(emb);
    const int32_t dstride = h->D, yoff = h->D / 2;     // channels per pixel; first channel of the y block
    const T *g = static_cast<const T *>(fg);
    // the test hook: the decode stops before launch fail_at, as if it had failed
    const int fail_at = h->fail_at;
    h->fail_at = -1;
    // A launch error is reported by the launch itself: the thread's last
    // error (possibly left by the caller's earlier HIP calls) is cleared
    // first and read after every launch.
    (void)hipGetLastError();
    // Launch i of the frame; with stage events on, the dispatch itself
    // records events 2i and 2i + 1 at the kernel's start and end.  Returns
    // false if the launch failed (or the test hook stops the frame here).
    auto launch = [&](int i, auto kernel, dim3 grid, dim3 block, size_t lds, auto... args) {
        if (i == fail_at) return false;
        if (h->stage_on)
            hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, stream, h->stage_ev[2 * i],
                                  h->stage_ev[2 * i + 1], 0u, args...);
        else
            hipLaunchKernelGGL(kernel, grid, block, lds, stream, args...);
        return hipGetLastError() == hipSuccess;
    };
    const bool mfma = Bw <= kMfmaBins && Bh <= kMfmaBins;     // the matrix-core assignment (and its peak prologue)
    // the frame's histogram set (clear) and the next frame's, whose first
    // nclear words an earlier frame may have written
    const int par = *sc.parity & 1;
    unsigned long long *hcur = sc.hrep + (size_t)par * sc.set_stride;
    unsigned long long *hnext = sc.hrep + (size_t)(1 - par) * sc.set_stride;
    const size_t nclear = sc.dirty[1 - par];
    const size_t nused = (size_t)kReplicas * nb;
    // once the clearing launch is enqueued: the other set is the next frame's
    auto flip = [&]() {
        sc.dirty[1 - par] = 0;
        *sc.parity = 1 - par;
    };
    constexpr int wpb = kVoteWpb<T, F>;
    const int64_t tiles = ((int64_t)npix + 31) / 32;
    int32_t *list = sc.list;
    int nslices, slice_px;
    const FusedPlan fp = fused_plan(npix);
    if (mfma && fp.ok) {
        // Two launches.  Launch 0 would be the compaction, which the vote
        // launch does itself here: its events record back to back.
        if (fail_at == 0) return CPE_ERR_HIP;
        if (h->stage_on) {
            if (hipEventRecord(h->stage_ev[0], stream) != hipSuccess ||
                hipEventRecord(h->stage_ev[1], stream) != hipSuccess)
                return CPE_ERR_HIP;
        }
        // launch 1: compaction of each workgroup's slices, recovery +
        // voting on them, the next frame's histograms cleared
        const FusedArgs fz{fg, fg_thr, fp.slice, fp.seg_cap, fp.rot, list, sc.counts, labels, score,
                           hnext, (int32_t)nclear};
        if (sc.dirty[par] < nused) sc.dirty[par] = nused;
        if (!launch(1, k_vote_mfma<T, F, false, true>, dim3(fp.grid), dim3(wpb * 64), 0, e, dstride, yoff,
                    (const int32_t *)nullptr, (const int32_t *)nullptr, 0, 0, npix, h->tb, Bw, Bh, hcur, cents,
                    h->cap, fz))
            return CPE_ERR_HIP;
        flip();
        nslices = fp.grid;             // the assignment reads the workgroups' segments as its slices
        slice_px = fp.seg_cap;
    } else {
        // launch 0: the participating pixels as a compact list (every pixel
        // when the frame has no foreground channel), the next frame's
        // histograms cleared
        const int64_t cg = ((int64_t)nclear + 255) / 256;
        const int clear_grid = cg < 1 ? 1 : cg > 64 ? 64 : (int)cg;
        nslices = slice_count(npix);
        slice_px = slice_pixels(npix);
        if (!g) list = nullptr;
        bool ok;
        if (!g)
            ok = launch(0, k_clear_u64, dim3(clear_grid), dim3(256), 0, hnext, (int32_t)nclear);
        else if (((uintptr_t)g & 15u) == 0)
            ok = launch(0, k_compact<T, true>, dim3(nslices), dim3(kCompactThreads), 0, g, npix, fg_thr, list,
                        sc.counts, labels, score, hnext, (int32_t)nclear);
        else
            ok = launch(0, k_compact<T, false>, dim3(nslices), dim3(kCompactThreads), 0, g, npix, fg_thr, list,
                        sc.counts, labels, score, hnext, (int32_t)nclear);
        if (!ok) return CPE_ERR_HIP;
        flip();
        // launch 1: recovery + voting, one pass per block of 32 x 32 bins;
        // grid: at most one workgroup per compute unit, no more waves than tiles
        const int64_t wgs = (tiles + wpb - 1) / wpb;
        const int grid = (int)(wgs < kVoteGrid ? wgs : kVoteGrid);
        auto vote_kernel = mfma ? k_vote_mfma<T, F, false, false> : k_vote_mfma<T, F, true, false>;
        if (sc.dirty[par] < nused) sc.dirty[par] = nused;
        if (!launch(1, vote_kernel, dim3(grid), dim3(wpb * 64), 0, e, dstride, yoff, (const int32_t *)list,
                    (const int32_t *)sc.counts, nslices, slice_px, npix, h->tb, Bw, Bh, hcur, cents, h->cap,
                    FusedArgs{}))
            return CPE_ERR_HIP;
    }
    if (mfma) {
        // launch 2: peak extraction in every workgroup's prologue, assignment
        constexpr int wpb2 = kAssignWpb<T, F>;
        const int64_t wgs2 = (tiles + wpb2 - 1) / wpb2;
        const int grid2 = (int)(wgs2 < kAssignGrid ? wgs2 : kAssignGrid);
        // labels only (no score map, no Eq8 threshold) on large frames: the
        // fast search, which pays off when every wave has several tiles (it
        // shortens each tile's work but lengthens its dependency chain)
        const bool labels_only = score == nullptr && !(fa.tau4096 < __builtin_inf());
        const bool fast = labels_only && (h->search_mode != 0 || (int64_t)npix >= kFastSearchPixels);
        auto assign_kernel = fast ? k_assign_mfma<T, F, true> : k_assign_mfma<T, F, false>;
        if (!launch(2, assign_kernel, dim3(grid2), dim3(wpb2 * 64), 0, e, dstride, yoff, (const int32_t *)list,
                    (const int32_t *)sc.counts, nslices, slice_px, npix, fa.tau4096, h->tb,
                    (const unsigned long long *)hcur, sc.hlast, Bw, Bh, cut, h->cap, cents, num, labels, score,
                    (int32_t)(h->search_mode == 1)))
            return CPE_ERR_HIP;
    } else {
        // launch 2 (larger grids): the stand-alone peak kernel, then the
        // generic assignment; the stage events bracket both (start of the
        // first, end of the second)
        if (fail_at == 2) return CPE_ERR_HIP;
        const PeakOut po{cents, num, sc.peaks, sc.kinfo};
        const size_t plds = (size_t)nb * 8 + (size_t)max_peaks(Bw, Bh) * 4;
        if (h->stage_on)
            hipExtLaunchKernelGGL(k_peaks, dim3(1), dim3(1024), (uint32_t)plds, stream, h->stage_ev[4], nullptr, 0u,
                                  (const unsigned long long *)hcur, sc.hlast, Bw, Bh, cut, h->cap, h->tb.cx,
                                  h->tb.cy, po);
        else
            hipLaunchKernelGGL(k_peaks, dim3(1), dim3(1024), plds, stream, (const unsigned long long *)hcur,
                               sc.hlast, Bw, Bh, cut, h->cap, h->tb.cx, h->tb.cy, po);
        if (hipGetLastError() != hipSuccess) return CPE_ERR_HIP;
        const size_t fixed2 = generic_assign_fixed(Bw, Bh, F, max_peaks(Bw, Bh));
        const int tp2 = pick_tile(fixed2, (size_t)Bw * 4, 120 * 1024);     // per pixel: its column distances
        const size_t lds2 = fixed2 + (size_t)Bw * tp2 * 4;
        const int64_t tiles2 = ((int64_t)npix + tp2 - 1) / tp2;
        const int grid2 = (int)(tiles2 < 2048 ? tiles2 : 2048);
        auto assign_kernel = k_assign_generic<T, F>;
        if (h->stage_on)
            hipExtLaunchKernelGGL(assign_kernel, dim3(grid2), dim3(tp2), (uint32_t)lds2, stream, nullptr,
                                  h->stage_ev[5], 0u, e, dstride, yoff, (const int32_t *)list,
                                  (const int32_t *)sc.counts, nslices, slice_px, npix, fa.tau4096, h->tb, Bw, Bh,
                                  (const int32_t *)sc.peaks, (const int32_t *)sc.kinfo, cents, labels, score);
        else
            hipLaunchKernelGGL(assign_kernel, dim3(grid2), dim3(tp2), lds2, stream, e, dstride, yoff,
                               (const int32_t *)list, (const int32_t *)sc.counts, nslices, slice_px, npix,
                               fa.tau4096, h->tb, Bw, Bh, (const int32_t *)sc.peaks, (const int32_t *)sc.kinfo, cents,
                               labels, score);
        if (hipGetLastError() != hipSuccess) return CPE_ERR_HIP;
    }
    return CPE_OK;
}


#define CPE_LAUNCH_RANGE(NAME, T, F0)                                       \
    cpe_status NAME(cpe_decoder *h, const Scratch &sc, const FrameArgs &a)  \
    {                                                                       \
        switch (h->F - (F0)) {                                              \
        case 0: return launch_all<T, (F0) + 0>(h, sc, a);                   \
        case 1: return launch_all<T, (F0) + 1>(h, sc, a);                   \
        case 2: return launch_all<T, (F0) + 2>(h, sc, a);                   \
        case 3: return launch_all<T, (F0) + 3>(h, sc, a);                   \
        case 4: return launch_all<T, (F0) + 4>(h, sc, a);                   \
        case 5: return launch_all<T, (F0) + 5>(h, sc, a);                   \
        case 6: return launch_all<T, (F0) + 6>(h, sc, a);                   \
        case 7: return launch_all<T, (F0) + 7>(h, sc, a);                   \
        default: return CPE_ERR_UNSUPPORTED;                                \
        }                                                                   \
    }

}  // namespace cpe
