/*
 * cpe_oracle.h -- CPU oracle of the sinusoidal-centroid-encoding decoder.
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, single-threaded, deliberately
 * slow reference used to check the GPU library.  It shares no source with
 * the GPU path (no headers, tables or helpers) and must never be linked into
 * the product.
 *
 * What it computes (Section 3.1 "Decoding Algorithm" and Section 3.2
 * "Decoding Implementation" of the paper):
 *   palettes P_w, P_h at the bin centres (Eq9), per-pixel per-axis distances
 *   to the palettes (Eq4 / Eq10), vote weights e^-d (Eq5), the vote
 *   histogram H = sum of E_x(a) E_y(b) over participating pixels (Eq6 /
 *   Eq11), strict 8-neighbour local maxima above a threshold (local-maxima
 *   search paragraph), nearest-candidate assignment (Eq7) and per-mask pixel
 *   counts (mask-aggregation paragraph).
 *
 * Two arithmetic modes:
 *   cpe_oracle_decode       canonical fixed-point arithmetic: inputs and
 *                           palettes rounded to 1/4096, exact integer
 *                           squared distances S, vote weights 2^15 e^-d of
 *                           the bucket given by the exponent and top 8
 *                           mantissa bits of fl32(S+1), exact 64-bit vote
 *                           sums; for the assignment the correctly rounded
 *                           binary32 distances sqrtf(fl32(S)) of both axes,
 *                           summed exactly.  Every discrete decision is
 *                           reproducible bit for bit by any correct
 *                           implementation.
 *   cpe_oracle_decode_real  the real-valued definition in fp64 with no
 *                           quantisation (diagnostic only).
 *
 * Parity pins: see the header of cpe_oracle.c.
 */
#ifndef CPE_ORACLE_H
#define CPE_ORACLE_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t bin_x, bin_y;   /* bin indices a_k, b_k                           */
    float x, y;             /* bin centre in pixels                           */
    double score;           /* vote mass H(a_k,b_k) * 2^-30                   */
    int32_t npix;           /* pixels assigned to this centroid               */
    int32_t reserved;       /* always 0                                       */
} cpe_oracle_centroid;      /* 32 bytes */

/* return codes */
#define CPE_ORACLE_OK 0
#define CPE_ORACLE_EINVAL 1

/* dtype: 0 = float32, 1 = float16 (IEEE binary16 bit patterns).
 * emb: [H][W][D] channels-last, D >= 4*n_freq and even: the x block is
 * channels [0, D/2), the y block [D/2, D), each (sin, cos) pairs of ascending
 * harmonics; the first 2*n_freq channels of each block are decoded (with
 * D > 4*n_freq only the low harmonics).  fg: [H][W]; both host memory.
 * Outputs (host): centroids[capacity], *num_centroids (true count K),
 * labels[H*W]; optional (may be NULL): score_map[H*W], hist[bins_h*bins_w]
 * (row-major [b][a]), pal_x[bins_w*2F], pal_y[bins_h*2F], weights[8192]
 * (indexed by the 8-bit bucket). */
int cpe_oracle_decode(int32_t H, int32_t W, int32_t D, int32_t dtype,
                      const void *emb, const void *fg,
                      const double *freq_x, const double *freq_y, int32_t n_freq,
                      int32_t bins_w, int32_t bins_h, int32_t capacity,
                      float fg_threshold, double peak_threshold,
                      cpe_oracle_centroid *centroids, int32_t *num_centroids,
                      int32_t *labels, float *score_map,
                      uint64_t *hist, int16_t *pal_x, int16_t *pal_y, uint16_t *weights);

/* The same with two of the paper's options:
 *   fg   may be NULL: then every pixel participates (the participating set of
 *        Section 3.1 is the whole output grid);
 *   tau  the mask threshold of Eq8 in distance units: a pixel keeps the label
 *        of its nearest candidate m only if D_m < 4096 tau, where D_m =
 *        sqrtf(S_x) + sqrtf(S_y) (exact sum) is its distance in units of
 *        1/4096; otherwise label 0, not counted.  +INFINITY keeps
 *        every participating pixel (cpe_oracle_decode); NaN is rejected. */
int cpe_oracle_decode_ex(int32_t H, int32_t W, int32_t D, int32_t dtype,
                         const void *emb, const void *fg,
                         const double *freq_x, const double *freq_y, int32_t n_freq,
                         int32_t bins_w, int32_t bins_h, int32_t capacity,
                         float fg_threshold, double peak_threshold, double tau,
                         cpe_oracle_centroid *centroids, int32_t *num_centroids,
                         int32_t *labels, float *score_map,
                         uint64_t *hist, int16_t *pal_x, int16_t *pal_y, uint16_t *weights);

/* Real-valued fp64 decoder (no quantisation, no threshold tau).  Outputs:
 * hist[bins_h*bins_w] (double), peak list (bin index b*bins_w+a, ascending)
 * in peaks[capacity] with *num_peaks = true count, labels[H*W]. */
int cpe_oracle_decode_real(int32_t H, int32_t W, int32_t D, int32_t dtype,
                           const void *emb, const void *fg,
                           const double *freq_x, const double *freq_y, int32_t n_freq,
                           int32_t bins_w, int32_t bins_h, int32_t capacity,
                           float fg_threshold, double peak_threshold,
                           double *hist, int32_t *peaks, int32_t *num_peaks,
                           int32_t *labels);

#ifdef __cplusplus
}
#endif
#endif
