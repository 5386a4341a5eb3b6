/*
 * cpe_decode.h -- C ABI of the MI355X (gfx950) decoder for sinusoidal
 * centroid positional encodings (instance segmentation).
 *
 * A frame is an H x W map of per-pixel embeddings T^ = concat(x^, y^)
 * (Section 3.1, Eq3) plus a foreground channel.  The decoder
 *   1. compares every foreground pixel's x^ and y^ with the encodings of the
 *      bin centres along each axis (palettes, Eq9; distances Eq4/Eq10),
 *   2. accumulates the soft votes e^-d into a B_w x B_h histogram (Eq5, Eq6,
 *      Eq11),
 *   3. extracts the bins that are strict 8-neighbour local maxima above a
 *      threshold and compacts them into a centroid list (local-maxima search
 *      paragraph of Section 3.2),
 *   4. assigns every foreground pixel to its nearest centroid in the encoded
 *      space (Eq7) and counts the pixels of each (mask-aggregation paragraph),
 *   5. writes an int32 label map (0 = background, k+1 = centroid k).
 *
 * Arithmetic.  All discrete decisions use a fixed-point arithmetic that any
 * correct implementation reproduces bit for bit:
 *   X = rint(4096 clamp(v, -1.5, 1.5)) per channel (a NaN clamps to -1.5):
 *   the input on a grid of 1/4096, in units of 1/4096;
 *   palettes P = rint(4096 gamma(bin centre)), bin centre (a+1) W/(B_w+1);
 *   S = |X - P|^2 exactly (integer);
 *   vote weight = rint(2^15 e^-d), d the distance at the centre of the
 *   bucket of S given by the exponent and top 8 mantissa bits of fl32(S+1);
 *   votes are exact 64-bit sums;
 *   assignment distance r = sqrtf(fl32(S)), the correctly rounded binary32
 *   square root (units of 1/4096); a pixel goes to the centroid with the
 *   smallest exact sum r_x + r_y, lowest index on ties.
 * Vote masses are reported as H * 2^-30 (so a pixel at distance 0 on both
 * axes adds 1.0).
 *
 * Layouts (all row-major, channels last):
 *   emb    [H][W][D]: channels [0,D/2) encode x, [D/2,D) encode y; within a
 *          block channel 2k = sin(w_k p), 2k+1 = cos(w_k p).  The decoder
 *          reads the first 2F channels of each block (F = n_freq; D = 4F
 *          reads them all)
 *   fg     [H][W], same dtype as emb; a pixel participates iff fg > threshold
 *   labels [H][W] int32
 *   score  [H][W] float (optional): expf(-(float)((r_x + r_y)/4096)) of the
 *          assigned centroid, 0 on unlabelled pixels
 *
 * Ownership.  The caller owns every buffer passed to cpe_decode (device
 * memory).  The handle owns the palettes, the table and all scratch; they
 * are allocated once in cpe_decode_create and freed by cpe_decode_destroy.
 * cpe_decode itself never allocates, never synchronises and never copies
 * to the host: it only enqueues work on `stream`.
 *
 * Errors.  Argument errors are detected on the host before any work is
 * enqueued and return CPE_ERR_INVALID_ARG.  A decode clears the calling
 * thread's last HIP error, then checks it after each of its launches: a
 * failed launch returns CPE_ERR_HIP at once (the frame's outputs are then
 * undefined).  No state carries over between frames -- a frame accumulates
 * its votes into one of two histogram sets, left clear by the frame before
 * it, and its first launch clears the other set for the next frame -- so the
 * next decode on the same handle is unaffected by a failed one.  Data-dependent outcomes (no centroid, more
 * centroids than the capacity) are reported through the device outputs,
 * never as errors.
 *
 * Threading.  A handle may be used by one stream at a time (its scratch is
 * per handle); separate handles are independent.
 */
#ifndef CPE_DECODE_H
#define CPE_DECODE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CPE_OK = 0,
    CPE_ERR_INVALID_ARG = 1,
    CPE_ERR_UNSUPPORTED = 2,
    CPE_ERR_OUT_OF_MEMORY = 3,
    CPE_ERR_HIP = 4
} cpe_status;

typedef enum { CPE_F32 = 0, CPE_F16 = 1 } cpe_dtype;

/* One decoded centroid (32 bytes). */
typedef struct {
    int32_t bin_x, bin_y; /* histogram bin (a_k, b_k)                               */
    float x, y;           /* bin centre in pixels: (a+1) W/(B_w+1), (b+1) H/(B_h+1)  */
    double score;         /* vote mass H(a_k, b_k) * 2^-30                           */
    int32_t npix;         /* number of pixels labelled k+1                           */
    int32_t reserved;     /* 0                                                       */
} cpe_centroid;

typedef struct cpe_decoder cpe_decoder;

/*
 * Build a decoder for frames of H x W pixels with D channels, decoding the
 * first n_freq harmonics of each axis.
 * Section 3.2 (Eq9): the palettes P_w, P_h are the encodings of the bin
 * centres; they are computed here once, on the host in fp64, and stay on the
 * device with the weight table for every later frame.
 *   out          receives the handle (set to NULL on failure)
 *   H, W         frame size, H*W <= 2^31 - 2^23 (2,139,095,040 pixels)
 *   D            channels per pixel: the x block is channels [0, D/2), the y
 *                block [D/2, D), each (sin, cos) pairs of ascending harmonics
 *                (Eq2, Eq3).  D = 4*n_freq decodes every harmonic.  D >
 *                4*n_freq decodes only the first n_freq of each block (the
 *                harmonics a coarse bin grid resolves; the palettes of Eq9 are
 *                built for those); then D must be even and each block 16-byte
 *                aligned (D * element size a multiple of 32), else
 *                CPE_ERR_UNSUPPORTED.  D < 4*n_freq or odd: CPE_ERR_INVALID_ARG
 *   dtype        element type of emb and fg
 *   freq_x/y     host arrays of n_freq angular frequencies in rad/pixel
 *                (harmonic k of the x and y encodings, k < n_freq), copied
 *   n_freq       1..16
 *   bins_w/h     1..128 histogram bins along x / y
 *   centroid_capacity  >= 1 and <= bins_w*bins_h; the number of centroid
 *                records cpe_decode may write.  ceil(B_w/2)*ceil(B_h/2) can
 *                never overflow (strict local maxima are pairwise
 *                non-adjacent).
 * Uses the current HIP device; the handle must be used on that device.
 * Returns CPE_ERR_INVALID_ARG, CPE_ERR_OUT_OF_MEMORY or CPE_ERR_HIP on failure.
 */
cpe_status cpe_decode_create(cpe_decoder **out, int32_t H, int32_t W, int32_t D, cpe_dtype dtype,
                             const double *freq_x, const double *freq_y, int32_t n_freq,
                             int32_t bins_w, int32_t bins_h, int32_t centroid_capacity);

/*
 * Decode one frame (Sections 3.1-3.2: Eq4-Eq7, local-maxima search, mask
 * aggregation), asynchronously on `stream`.
 *   emb, fg        device inputs, layouts above; emb 16-byte aligned, fg
 *                  aligned to its element size
 *   H, W           must equal the values given to cpe_decode_create
 *   fg_threshold   pixel p votes and is labelled iff (float)fg[p] > fg_threshold
 *   peak_threshold a bin can be a centroid only if its vote mass exceeds this
 *                  (compared as H > floor(peak_threshold * 2^30))
 *   centroids      device [centroid_capacity]: records 0..min(K,cap)-1 are
 *                  written, in ascending bin order b*B_w + a
 *   num_centroids  device int32: the true number K of local maxima (may
 *                  exceed the capacity; then only the first cap are used)
 *   labels         device [H][W] int32, 16-byte aligned
 *   score_map      device [H][W] float or NULL
 * Non-finite thresholds are rejected.
 */
cpe_status cpe_decode(cpe_decoder *h, hipStream_t stream, const void *emb, const void *fg,
                      int32_t H, int32_t W, float fg_threshold, double peak_threshold,
                      cpe_centroid *centroids, int32_t *num_centroids, int32_t *labels,
                      float *score_map);

/* Options of cpe_decode_ex. */
typedef struct {
    float fg_threshold;     /* as in cpe_decode; unused when fg is NULL          */
    int32_t reserved;       /* must be 0                                         */
    double peak_threshold;  /* as in cpe_decode                                  */
    double tau;             /* Eq8 mask threshold in distance units; +INFINITY:
                               none (every participating pixel is labelled)     */
} cpe_decode_options;

/*
 * cpe_decode with the two options of Section 3.1 that the foreground channel
 * otherwise replaces:
 *   fg == NULL   every pixel of the frame participates (the participating set
 *                of Eq6 is the whole output grid); otherwise as cpe_decode.
 *   opt->tau     Eq8: a participating pixel keeps the label of its nearest
 *                candidate m (Eq7) only if that distance is below tau, the
 *                distance being the exact sum D_m = r_x + r_y of the two axis
 *                distances in units of 1/4096 (test: D_m < 4096 tau in
 *                binary64, strict).  A pixel
 *                that fails gets label 0 and score 0 and is not counted in
 *                npix.  tau <= 0 labels nothing; +INFINITY is cpe_decode.
 * The histogram and the centroid records do not depend on tau.
 * Errors as cpe_decode; NaN or -INFINITY tau, a non-finite threshold or a
 * nonzero reserved field is CPE_ERR_INVALID_ARG.
 */
cpe_status cpe_decode_ex(cpe_decoder *h, hipStream_t stream, const void *emb, const void *fg,
                         int32_t H, int32_t W, const cpe_decode_options *opt,
                         cpe_centroid *centroids, int32_t *num_centroids, int32_t *labels,
                         float *score_map);

/*
 * cpe_decode_ex for callers that cannot allocate device memory around a
 * decode (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same frame, arguments, outputs and errors as
 * cpe_decode_ex, and the handle's constants, but the per-frame scratch (vote
 * histograms, participating-pixel list, slice counts, peak list) is a static
 * device array of the library, about 9.7 MB, held by each device the
 * library runs on until the process ends, instead of the handle's.  The
 * call itself allocates nothing.
 *   Limit: frames of at most 2,097,152 pixels (H*W <= 2^21, e.g. 1024 x
 *   2048); a handle for a larger frame gets CPE_ERR_UNSUPPORTED.  The
 *   array's device address is looked up by cpe_decode_create on its device;
 *   if that lookup failed the call returns CPE_ERR_HIP.
 *   Every call on a device shares that device's array: calls that overlap in
 *   time on one device (other streams, other threads, other handles) race
 *   and give undefined results; calls ordered on one stream are safe, since
 *   each frame finds the histograms it accumulates into clear and clears
 *   those of the next call, whatever its handle.
 *   cpe_decode_get_histogram does not see these frames (it returns the
 *   handle's latest cpe_decode / cpe_decode_ex frame).
 */
cpe_status cpe_decode_noalloc(cpe_decoder *h, hipStream_t stream, const void *emb, const void *fg,
                              int32_t H, int32_t W, const cpe_decode_options *opt,
                              cpe_centroid *centroids, int32_t *num_centroids, int32_t *labels,
                              float *score_map);

/*
 * Binary instance masks M^_m of Eq8 from a label map written by cpe_decode or
 * cpe_decode_ex on this handle, asynchronously on `stream`:
 *   masks[m][p] = 1 if labels[p] == first + m + 1, else 0,
 * for m = 0 .. count-1 and p = 0 .. H*W-1, one byte per pixel, mask m at
 * byte offset m*H*W.  Mask m belongs to centroid first+m, i.e. to bin
 * (bin_x, bin_y) of that record; indices at or past min(K, cap) give empty
 * masks.  (The paper preallocates one mask per histogram bin; placing the
 * masks of this call at slot bin_y*B_w + bin_x gives that layout.)
 *   labels  device [H][W] int32, 16-byte aligned (caller-owned)
 *   masks   device [count][H][W] uint8, 16-byte aligned (caller-owned)
 *   first   >= 0; count >= 1; first + count <= centroid_capacity
 * Errors: CPE_ERR_INVALID_ARG for a bad argument (before any work is
 * enqueued), CPE_ERR_HIP for a failed launch.
 */
cpe_status cpe_decode_masks(cpe_decoder *h, hipStream_t stream, const int32_t *labels, int32_t H, int32_t W,
                            int32_t first, int32_t count, uint8_t *masks);

/* Release a decoder (waits for nothing; the caller must have synchronised
 * the streams that used it).  NULL is a no-op. */
cpe_status cpe_decode_destroy(cpe_decoder *h);

/* Static string describing a status code. */
const char *cpe_status_string(cpe_status s);

/*
 * Inspection (tests and profiling).  Host copies of the constants built by
 * cpe_decode_create: pal_x [bins_w][2F] and pal_y [bins_h][2F] int16 (Eq9
 * palettes x4096, rounded), weights [8192] uint16 (2^15 e^-d per 8-bit
 * bucket).  Any pointer may be NULL.
 */
cpe_status cpe_decode_get_tables(const cpe_decoder *h, int16_t *pal_x, int16_t *pal_y, uint16_t *weights);

/*
 * Enqueue on `stream` a device-to-device copy of the vote histogram of the
 * most recent cpe_decode on this handle (Eq6/Eq11 in fixed point): [bins_h]
 * [bins_w] uint64, entry [b][a] = sum over foreground pixels of
 * q_x(a) q_y(b).
 */
cpe_status cpe_decode_get_histogram(cpe_decoder *h, hipStream_t stream, uint64_t *hist);

/*
 * Self-check (tests): enqueue on `stream` a comparison of the square root the
 * assignment uses (the hardware square root plus a rounding correction) with
 * the IEEE correctly rounded sqrtf on every binary32 value it can receive
 * (0 and every float in [1, 2^32)); the device uint64 *mismatches (8-byte
 * aligned, caller-owned) receives the number of differing results, 0 when
 * the assignment's distances are exactly those of Eq4 as defined above.
 */
cpe_status cpe_check_sqrt(hipStream_t stream, unsigned long long *mismatches);

/*
 * Testing: make the next decode on this handle stop before its launch
 * `launch` (0, 1 or 2, numbered as for cpe_decode_set_stage_events; -1
 * cancels) and return CPE_ERR_HIP as if that launch had failed; the earlier
 * launches of that frame are enqueued (none before launch 1 in a two-launch
 * frame).  One-shot.
 */
cpe_status cpe_decode_test_fail_launch(cpe_decoder *h, int32_t launch);

/*
 * Testing: the assignment search of later label-only decodes on this handle
 * (no score map, tau = +inf, grids up to 32 x 32 bins).  mode 0 (default):
 * the fast search (hardware square roots, near ties recomputed exactly) on
 * frames of at least 2^20 pixels, the exact search on smaller ones; 1: the
 * fast-search kernel at any size with every tile treated as a near tie,
 * i.e. recomputed with correctly rounded distances and the exact search;
 * 2: the fast search at any size.  The labels are the same in every mode.
 * CPE_ERR_INVALID_ARG for another mode.
 */
cpe_status cpe_decode_test_search_mode(cpe_decoder *h, int32_t mode);

/* Bytes of device memory the handle holds (constants + scratch). */
size_t cpe_decode_workspace_bytes(const cpe_decoder *h);

/*
 * Kernels each frame of this handle launches: 2 when the vote launch also
 * lists the participating pixels (frames of up to 2^21 pixels on grids up to
 * 32 x 32 bins), else 3 (numbered as for cpe_decode_set_stage_events); 0 for
 * NULL.
 */
int32_t cpe_decode_launch_count(const cpe_decoder *h);

/*
 * Profiling: when `events` is non-NULL, every later cpe_decode on this handle
 * launches its i-th kernel (i = 0, 1, 2) so that the dispatch itself records
 * events[2i] when the kernel starts and events[2i+1] when it ends, on the
 * decode's stream; hipEventElapsedTime(events[2i], events[2i+1]) is then that
 * kernel's duration: 0 = compaction of the participating pixels and
 * clearing of the next frame's vote histograms (only the clearing without a
 * foreground channel), 1 = recovery + voting, 2 = peak extraction +
 * assignment (one kernel for grids up to 32 x 32 bins; above, events 4 and 5
 * bracket the peak kernel and the assignment kernel that follows it).
 * Frames of up to 2^21 pixels on grids up to 32 x 32 bins take two
 * launches: kernel 1 also compacts and clears, and events 0 and 1 are
 * recorded back to back, with no kernel between them.  `n_events` must be
 * CPE_STAGE_EVENTS;
 * the caller owns the events and must keep them alive while set.  NULL
 * switches the recording off.
 */
#define CPE_STAGE_EVENTS 6
cpe_status cpe_decode_set_stage_events(cpe_decoder *h, hipEvent_t *events, int32_t n_events);

/*
 * Ablation, not the decoder: the per-tuple GPU decoder of the prior work the
 * paper compares against (Section 3.2 "Histogram Accumulation" and "Mask
 * Aggregation"; Table 3, "Naive"), with the real-valued definition of
 * Section 3.1 in fp32 and no quantisation:
 *   votes   one thread per (pixel, bin) tuple computes both distances to the
 *           real palettes gamma(bin centre) and adds e^-d_x e^-d_y to
 *           H(a, b) with a float atomicAdd (Eq4, Eq6).  The addition order,
 *           and so the last bits of H, differ from run to run;
 *   peaks   strict 8-neighbour maxima with H > peak_threshold, in bin order;
 *   labels  one thread per (pixel, candidate) tuple recomputes the affinity
 *           e^-d_x e^-d_y; each pixel takes the largest, lowest index on
 *           equal affinities (Eq7); counts in the records.
 * Same handle and arguments as cpe_decode (fg required; emb and fg aligned
 * to their element size, labels to 4 bytes; peak_threshold in vote-mass
 * units, H itself here), plus
 *   hist   device [B_h][B_w] float: receives H, or NULL.
 * The records' score is H(a_k, b_k).  Results agree with the real-valued
 * definition (fp64) to fp32 rounding; near-equal distances and near-equal
 * neighbouring bins may decide differently, and repeated calls may differ
 * in those decisions.  The first call allocates the ablation's workspace
 * (real palettes, histogram, peak list, one 64-bit key per pixel), freed by
 * cpe_decode_destroy; the call is otherwise asynchronous on `stream`.  Not
 * for use with cpe_decode on overlapping streams.
 */
cpe_status cpe_decode_naive(cpe_decoder *h, hipStream_t stream, const void *emb, const void *fg,
                            int32_t H, int32_t W, float fg_threshold, double peak_threshold,
                            cpe_centroid *centroids, int32_t *num_centroids, int32_t *labels, float *hist);

#ifdef __cplusplus
}
#endif
#endif /* CPE_DECODE_H */
