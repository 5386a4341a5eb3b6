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
// Nothing in it carries over from one frame to the next: the first launch of
// every frame clears the vote histograms.
struct Scratch {
    unsigned long long *hrep;    // [kReplicas][nb] vote histograms
    unsigned long long *hlast;   // [nb] summed histogram of the frame
    int32_t *peaks;              // [cap] a | b << 16 (generic path)
    int32_t *kinfo;              // [0] = min(K, cap), [1] = K (generic path)
    int32_t *counts;             // [kMaxSlices] entries per slice of the participating-pixel list
    int32_t *list;               // participating pixels, in slices: H*W + one slice
};

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
    int fail_at;                         // test hook: the next decode stops before this launch (-1: none)
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
