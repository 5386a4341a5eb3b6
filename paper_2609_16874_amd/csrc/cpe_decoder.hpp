// cpe_decoder.hpp -- the decoder handle and the launch sequence of one frame
// (private to the library).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "cpe_common.hpp"

namespace cpe {

// Per-frame scratch of the launch sequence: everything a decode writes and
// reads besides the caller's inputs and outputs and the handle's constants.
// The vote histograms come in two sets of set_stride words each.  A frame
// accumulates into set *parity, which is clear when the frame starts, and
// its first launch that runs clears the first dirty[1 - *parity] words of
// the other set (the ones an earlier frame may have written); *parity flips
// once that launch is enqueued.  So every frame starts on a clear set, also
// after a decode that failed part-way.
struct Scratch {
    unsigned long long *hrep;    // [2][set_stride]: per set [kReplicas][nb] vote histograms
    size_t set_stride;           // words per set (>= kReplicas * nb)
    int *parity;                 // host: the set of the next frame (0 or 1)
    size_t *dirty;               // host: [2] leading words of each set that may be nonzero
    unsigned long long *hlast;   // [nb] summed histogram of the frame
    int32_t *peaks;              // [cap] a | b << 16 (generic path)
    int32_t *kinfo;              // [0] = min(K, cap), [1] = K (generic path)
    int32_t *counts;             // [kMaxSlices] entries per slice of the participating-pixel list
    int32_t *list;               // participating pixels, in slices (list_entries() in cpe_decode.hip)
};

// The folded compaction's plan for a frame of npix pixels (FusedArgs in
// k_mfma.hpp): `grid` workgroups, each voting on slices of `slice` pixels
// dealt to it in turn and listing a range of seg_cap pixels (a multiple of
// 8) for the assignment; ok = false when the frame is too large.
struct FusedPlan {
    bool ok;
    int slice, grid, seg_cap, rot;
};
inline FusedPlan fused_plan(int64_t npix)
{
    FusedPlan fp{false, 64, 1, 64, 0};
    if (npix < 1 || npix > kFusedMaxPixels) return fp;
    // 64-pixel slices (one wave step) dealt in turn.  When a workgroup owns
    // 4096 pixels or more, consecutive workgroups' slices would form
    // columns of the frame (at 1024 x 2048: 64-pixel strips, 8 rows apart),
    // whose foreground counts differ much: there the slices are dealt with a
    // rotation of 37 per round when the rounds are whole, else they are of
    // 1024 pixels (on the seeded 1024 x 2048 frame of 150 instances the
    // largest workgroup share of the foreground is 1.051 times the mean with
    // the rotation, 1.091 with 1024-pixel slices and 1.29 with neither)
    const int64_t per_wg = (npix + kMaxSlices - 1) / kMaxSlices;
    int slice = 64, rot = 0;
    if (per_wg >= 4096) {
        if (((npix + 63) / 64) % kMaxSlices == 0)
            rot = 37;
        else
            slice = 1024;
    }
    const int64_t nsl = (npix + slice - 1) / slice;
    const int64_t grid = nsl < kMaxSlices ? nsl : kMaxSlices;
    if ((nsl + grid - 1) / grid * slice > kFusedMaxSeg) return fp;     // the vote's list in LDS
    const int64_t seg = ((npix + grid - 1) / grid + 7) / 8 * 8;
    return FusedPlan{true, slice, (int)grid, (int)seg, rot};
}

}  // namespace cpe

struct cpe_decoder {
    int32_t H, W, D, F, bins_w, bins_h, cap;
    cpe_dtype dtype;
    int device;
    std::vector<int16_t> pal_x, pal_y;   // host copies, [bins][2F]
    std::vector<uint16_t> wt;            // host copy of the weight buckets (bucket order)
    unsigned char *dev;                  // single device allocation
    size_t dev_bytes;
    cpe::Tables tb;
    cpe::Scratch sc;                     // per-frame scratch, in the device allocation
    int parity;                          // histogram set of the next frame (sc.parity points here)
    size_t dirty[2];                     // words of each set that may be nonzero (sc.dirty points here)
    int fail_at;                         // test hook: the next decode stops before this launch (-1: none)
    int search_mode;                     // test hook: 0 default, 1 every tile exact, 2 fast search at any size
    hipEvent_t stage_ev[CPE_STAGE_EVENTS];
    bool stage_on;
    // per-tuple ablation (cpe_decode_naive): real palettes gamma(bin centre)
    // in fp32, [bins][2F], and its device workspace, allocated on first use
    std::vector<float> palf_x, palf_y;
    unsigned char *naive = nullptr;
    size_t naive_bytes = 0;
};

namespace cpe {

// Arguments of one frame's launch sequence.
struct FrameArgs {
    hipStream_t stream;
    const void *emb, *fg;
    float fg_thr;
    long long cut;               // floor(peak_threshold * 2^30), saturated
    double tau4096;              // a pixel is labelled iff its distance sum < 4096 tau (Eq8)
    cpe_centroid *cents;
    int32_t *num, *labels;
    float *score;
};

// Enqueue the kernels of one frame for element type T and F harmonics, with
// the per-frame scratch sc; each is defined in one of the launch_*.hip
// translation units.
cpe_status launch_f32_lo(cpe_decoder *h, const Scratch &sc, const FrameArgs &a);   // F = 1..8
cpe_status launch_f32_hi(cpe_decoder *h, const Scratch &sc, const FrameArgs &a);   // F = 9..16
cpe_status launch_f16_lo(cpe_decoder *h, const Scratch &sc, const FrameArgs &a);
cpe_status launch_f16_hi(cpe_decoder *h, const Scratch &sc, const FrameArgs &a);

// Enqueue the binary masks of centroids first .. first+count-1 (masks.hip).
cpe_status launch_masks(hipStream_t stream, const int32_t *labels, int64_t npix, int32_t first, int32_t count,
                        uint8_t *masks);

}  // namespace cpe
