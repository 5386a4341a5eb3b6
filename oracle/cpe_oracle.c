/*
 * cpe_oracle.c -- plain CPU oracle of the centroid-encoding decoder.
 *
 * TEST INFRASTRUCTURE ONLY (see cpe_oracle.h).  Single-threaded, no SIMD, no
 * blocking, no reordering beyond what each step's definition states.  Built
 * with gcc -O2 and without -ffast-math so that rintf, sqrtf and the (float)
 * casts are the IEEE round-to-nearest-even operations the canonical
 * arithmetic names.
 *
 * The steps follow Section 3 of the paper in its own order:
 *   palettes (Eq9)                     -> build_palette()
 *   per-axis distances, weights        -> axis_profile()      (Eq4, Eq5, Eq10)
 *   vote histogram                     -> accumulate over S   (Eq6, Eq11)
 *   local-maxima search                -> is_peak()           (LMS paragraph)
 *   assignment and counts              -> assignment loop     (Eq7, mask
 *                                                              aggregation)
 *
 * Canonical arithmetic (the reading adopted where the paper fixes no
 * precision; every constant below is part of that contract):
 *   bin centres   x_a = (a+1) W / (B_w+1), y_b = (b+1) H / (B_h+1)  (fp64;
 *                 Eq9 with u = 2x/W - 1 and continuous pixel coordinates)
 *   palette       P[a][2k] = rint(4096 sin(w_k x_a)), P[a][2k+1] =
 *                 rint(4096 cos(w_k x_a)), fp64, stored as int16
 *   input         X = rintf(4096.0f * clamp(v, -1.5, 1.5)) in fp32 (a NaN
 *                 channel clamps to -1.5): the input on the palette's grid
 *                 of 1/4096
 *   participation p in S  <=>  (float)fg(p) > fg_threshold; with no fg
 *                 channel every pixel is in S (the set of Section 3.1)
 *   distance      S_x = sum_c (X_c - P[a][c])^2 (exact integer, < 2^32)
 *   weight        with u = fl32(S+1) = 2^e (1 + f), 0 <= f < 1, the 8-bit
 *                 bucket of S is key(S) = e 2^8 + floor(f 2^8) (exponent and
 *                 top 8 mantissa bits of u); q = WT[key] = rint(2^15 e^-d~),
 *                 d~ = sqrt(2^e (1 + (t+0.5)/2^8) - 1)/4096 the distance at
 *                 the bucket centre, t = key mod 2^8 (0 for S = 0)  (Eq5/Eq10)
 *   votes         H[b][a] = sum_{p in S} q_x(p,a) q_y(p,b)  (exact uint64)
 *   peaks         H[b][a] > floor(theta_peak 2^30) and > every in-range
 *                 8-neighbour; listed in ascending b*B_w + a
 *   distance      r = sqrtf(fl32(S)), the correctly rounded binary32 square
 *   (Eq7)         root of S rounded to binary32: the Euclidean distance in
 *                 units of 1/4096
 *   assignment    D_k = r_x(a_k) + r_y(b_k), the exact sum (representable in
 *                 binary64); the smallest k with the minimal D_k wins;
 *                 label = k+1, background 0
 *   mask test     (Eq8) the winner m keeps the pixel only if D_m < 4096 tau
 *                 (binary64 compare; tau = +inf keeps every pixel of S); a
 *                 pixel that fails it gets label 0 and is not counted
 *   score map     expf(-(float)(D_m / 4096)) for labelled pixels
 *
 * Pins (tests/test_oracle_*.py), each independent of this file's code:
 *   - weight buckets against e^-d over each bucket's exact range; palette
 *     sin^2+cos^2 = 1 and its values against gamma at the centres;
 *   - the vote histogram against the paper's matrix form E_x^T E_y in fp64
 *     (numpy), within the quantisation error bound;
 *   - brute force on tiny frames: exhaustive scan of every grid position for
 *     the peaks and every candidate for each pixel's assignment, with exact
 *     rational sums of the square roots;
 *   - noise-free frames whose centroids sit on bin centres decode to the
 *     generating centroids and the generating label map;
 *   - invariants: labels partition the foreground, counts sum to |S|,
 *     peaks pairwise non-adjacent, instance-order independence;
 *   - the assignment against Eq7 evaluated in fp64 on the unquantised input
 *     (at most 0.1 % of the foreground differs on the 256x256, 640x640 and
 *     1024x2048 workloads, all of them near-ties);
 *   - the Eq8 mask threshold and the all-pixels mode: the exhaustive search,
 *     a noise-free frame where a small tau keeps exactly the instance
 *     pixels, and nesting in tau;
 *   - the fp64 real-valued mode: its histogram against E_x^T E_y, its peaks
 *     against a library maximum filter, its labels against a numpy argmin.
 * The whole pipeline against the paper's own decoder: parity unpinned (no
 * implementation or worked example is published).
 */
#include "cpe_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define FIX_SCALE 4096.0f       /* input, palette and distance fixed point   */
#define V_CLAMP 1.5f            /* inputs are clamped to [-1.5, 1.5]         */
#define W_MANT 8                /* mantissa bits of fl32(S+1): weight bucket */
#define W_KEYS (32 << W_MANT)   /* 32 binades of S+1 in [1, 2^32)            */

/* IEEE binary16 -> binary32, exact (every half is a float). */
static float half_to_float(uint16_t h)
{
    uint32_t sign = (uint32_t)(h >> 15) & 1u;
    uint32_t expo = (uint32_t)(h >> 10) & 0x1fu;
    uint32_t mant = (uint32_t)h & 0x3ffu;
    float mag;
    if (expo == 0) {
        mag = ldexpf((float)mant, -24);                 /* zero / subnormal */
    } else if (expo == 31) {
        mag = mant ? NAN : INFINITY;
    } else {
        mag = ldexpf((float)(mant | 0x400u), (int)expo - 25);
    }
    return sign ? -mag : mag;
}

static float load_value(const void *base, int32_t dtype, size_t index)
{
    if (dtype == 0) return ((const float *)base)[index];
    return half_to_float(((const uint16_t *)base)[index]);
}

/* Input to fixed point: clamp to [-1.5, 1.5] (NaN -> -1.5), round to the
 * nearest multiple of 1/4096 (ties to even), in units of 1/4096. */
static int32_t to_fixed(float v)
{
    float c = v;
    if (isnan(c) || c < -V_CLAMP) c = -V_CLAMP;
    if (c > V_CLAMP) c = V_CLAMP;
    return (int32_t)rintf(FIX_SCALE * c);
}

/* m-bit distance bucket of an exact squared distance S: the exponent and
 * the top m mantissa bits of the binary32 value of S+1. */
static int32_t dist_key(uint32_t S, int32_t m)
{
    float u = (float)(uint32_t)(S + 1u);
    uint32_t bits;
    memcpy(&bits, &u, sizeof bits);
    return (int32_t)(bits >> (23 - m)) - (127 << m);
}

/* Bucket centre expressed as a distance in embedding units. */
static double key_distance(int32_t key, int32_t m)
{
    if (key == 0) return 0.0;
    const int32_t e = key >> m, t = key & ((1 << m) - 1);
    const double s_mid = ldexp(1.0 + ((double)t + 0.5) / (double)(1 << m), e) - 1.0;
    return sqrt(s_mid) / 4096.0;
}

/* Eq9: palette of n bins along an axis of `extent` pixels, 2F channels. */
static void build_palette(int32_t n, int32_t extent, const double *freq, int32_t F, int16_t *pal)
{
    for (int32_t a = 0; a < n; a++) {
        double centre = ((double)(a + 1) * (double)extent) / (double)(n + 1);
        for (int32_t k = 0; k < F; k++) {
            double phase = freq[k] * centre;
            pal[a * 2 * F + 2 * k] = (int16_t)rint(4096.0 * sin(phase));
            pal[a * 2 * F + 2 * k + 1] = (int16_t)rint(4096.0 * cos(phase));
        }
    }
}

/* Eq5 weights e^-d of the 8-bit buckets. */
static void build_weights(uint16_t *wt)
{
    for (int32_t key = 0; key < W_KEYS; key++) wt[key] = (uint16_t)rint(32768.0 * exp(-key_distance(key, W_MANT)));
}

/* Eq4/Eq10 for one axis of one pixel: the exact squared distance S to every
 * palette entry, giving its vote weight q[a] (from the bucket of S) and its
 * distance r[a] = sqrtf(fl32(S)) in units of 1/4096. */
static void axis_profile(const int32_t *X, const int16_t *pal, int32_t n, int32_t twoF,
                         const uint16_t *wt, uint32_t *q, float *r)
{
    for (int32_t a = 0; a < n; a++) {
        uint64_t s = 0;
        for (int32_t ch = 0; ch < twoF; ch++) {
            int64_t diff = (int64_t)X[ch] - (int64_t)pal[a * twoF + ch];
            s += (uint64_t)(diff * diff);
        }
        if (q) q[a] = wt[dist_key((uint32_t)s, W_MANT)];
        if (r) r[a] = sqrtf((float)(uint32_t)s);
    }
}

static int64_t peak_cut(double theta)
{
    double t = floor(theta * 1073741824.0);
    if (t < -1.0) return -1;
    if (t > 4.0e18) return (int64_t)4000000000000000000LL;
    return (int64_t)t;
}

static int check_args(int32_t H, int32_t W, int32_t D, int32_t dtype, const void *emb,
                      const double *fx, const double *fy, int32_t n_freq, int32_t bw, int32_t bh,
                      int32_t cap, float fg_thr, double peak_thr)
{
    if (H < 1 || W < 1 || (int64_t)H * (int64_t)W > 2147483647LL) return CPE_ORACLE_EINVAL;
    /* D channels per pixel: the x block [0, D/2) and the y block [D/2, D),
     * each (sin, cos) pairs of ascending harmonics (Eq2, Eq3); the decoder
     * uses the first 2 n_freq channels of each block (D > 4 n_freq: only the
     * low harmonics, those a coarse bin grid resolves) */
    if (n_freq < 1 || n_freq > 16 || D < 4 * n_freq || D % 2 != 0) return CPE_ORACLE_EINVAL;
    if (dtype != 0 && dtype != 1) return CPE_ORACLE_EINVAL;
    if (!emb || !fx || !fy) return CPE_ORACLE_EINVAL;
    if (bw < 1 || bw > 128 || bh < 1 || bh > 128 || cap < 1) return CPE_ORACLE_EINVAL;
    if (isnan(fg_thr) || isnan(peak_thr)) return CPE_ORACLE_EINVAL;
    return CPE_ORACLE_OK;
}

/* strict 8-neighbour local maximum of a [bh][bw] map; out-of-range ignored */
static int is_peak_u64(const uint64_t *h, int32_t bw, int32_t bh, int32_t a, int32_t b)
{
    uint64_t v = h[b * bw + a];
    for (int32_t db = -1; db <= 1; db++)
        for (int32_t da = -1; da <= 1; da++) {
            if (!da && !db) continue;
            int32_t nb = b + db, na = a + da;
            if (nb < 0 || nb >= bh || na < 0 || na >= bw) continue;
            if (!(v > h[nb * bw + na])) return 0;
        }
    return 1;
}

static int is_peak_f64(const double *h, int32_t bw, int32_t bh, int32_t a, int32_t b)
{
    double v = h[b * bw + a];
    for (int32_t db = -1; db <= 1; db++)
        for (int32_t da = -1; da <= 1; da++) {
            if (!da && !db) continue;
            int32_t nb = b + db, na = a + da;
            if (nb < 0 || nb >= bh || na < 0 || na >= bw) continue;
            if (!(v > h[nb * bw + na])) return 0;
        }
    return 1;
}

/* p in S: the foreground test, or every pixel when there is no fg channel */
static int participates(const void *fg, int32_t dtype, size_t p, float fg_threshold)
{
    return !fg || load_value(fg, dtype, p) > fg_threshold;
}

int cpe_oracle_decode(int32_t H, int32_t W, int32_t D, int32_t dtype,
                      const void *emb, const void *fg,
                      const double *freq_x, const double *freq_y, int32_t n_freq,
                      int32_t bins_w, int32_t bins_h, int32_t capacity,
                      float fg_threshold, double peak_threshold,
                      cpe_oracle_centroid *centroids, int32_t *num_centroids,
                      int32_t *labels, float *score_map,
                      uint64_t *hist, int16_t *pal_x, int16_t *pal_y, uint16_t *wt_out)
{
    if (!fg) return CPE_ORACLE_EINVAL;
    return cpe_oracle_decode_ex(H, W, D, dtype, emb, fg, freq_x, freq_y, n_freq, bins_w, bins_h, capacity,
                                fg_threshold, peak_threshold, INFINITY, centroids, num_centroids, labels,
                                score_map, hist, pal_x, pal_y, wt_out);
}

int cpe_oracle_decode_ex(int32_t H, int32_t W, int32_t D, int32_t dtype,
                         const void *emb, const void *fg,
                         const double *freq_x, const double *freq_y, int32_t n_freq,
                         int32_t bins_w, int32_t bins_h, int32_t capacity,
                         float fg_threshold, double peak_threshold, double tau,
                         cpe_oracle_centroid *centroids, int32_t *num_centroids,
                         int32_t *labels, float *score_map,
                         uint64_t *hist, int16_t *pal_x, int16_t *pal_y, uint16_t *wt_out)
{
    if (check_args(H, W, D, dtype, emb, freq_x, freq_y, n_freq, bins_w, bins_h, capacity,
                   fg_threshold, peak_threshold) != CPE_ORACLE_OK ||
        isnan(tau) || !centroids || !num_centroids || !labels)
        return CPE_ORACLE_EINVAL;

    const int32_t F = n_freq, twoF = 2 * n_freq, yoff = D / 2;
    const size_t npix = (size_t)H * (size_t)W;
    const int32_t nbins = bins_w * bins_h;

    int16_t *Pw = malloc(sizeof(int16_t) * bins_w * twoF);
    int16_t *Ph = malloc(sizeof(int16_t) * bins_h * twoF);
    uint16_t *wt = malloc(sizeof(uint16_t) * W_KEYS);
    uint64_t *Hv = calloc((size_t)nbins, sizeof(uint64_t));
    int32_t *X = malloc(sizeof(int32_t) * twoF);
    int32_t *Y = malloc(sizeof(int32_t) * twoF);
    float *rx = malloc(sizeof(float) * bins_w), *ry = malloc(sizeof(float) * bins_h);
    uint32_t *qx = malloc(sizeof(uint32_t) * bins_w), *qy = malloc(sizeof(uint32_t) * bins_h);
    int32_t *peak_a = malloc(sizeof(int32_t) * nbins), *peak_b = malloc(sizeof(int32_t) * nbins);

    /* palettes, preloaded once (Section 3.2, Eq9), and the weight buckets */
    build_palette(bins_w, W, freq_x, F, Pw);
    build_palette(bins_h, H, freq_y, F, Ph);
    build_weights(wt);

    /* histogram accumulation: H(a,b) = sum_{p in S} E_x(p,a) E_y(p,b) */
    for (size_t p = 0; p < npix; p++) {
        if (!participates(fg, dtype, p, fg_threshold)) continue;
        for (int32_t c = 0; c < twoF; c++) {
            X[c] = to_fixed(load_value(emb, dtype, p * (size_t)D + (size_t)c));
            Y[c] = to_fixed(load_value(emb, dtype, p * (size_t)D + (size_t)(yoff + c)));
        }
        axis_profile(X, Pw, bins_w, twoF, wt, qx, NULL);
        axis_profile(Y, Ph, bins_h, twoF, wt, qy, NULL);
        for (int32_t b = 0; b < bins_h; b++)
            for (int32_t a = 0; a < bins_w; a++)
                Hv[b * bins_w + a] += (uint64_t)qx[a] * (uint64_t)qy[b];
    }

    /* local-maxima search, candidates listed in ascending bin index */
    const int64_t cut = peak_cut(peak_threshold);
    int32_t K = 0;
    for (int32_t b = 0; b < bins_h; b++)
        for (int32_t a = 0; a < bins_w; a++) {
            int64_t v = (int64_t)Hv[b * bins_w + a];
            if (v > cut && is_peak_u64(Hv, bins_w, bins_h, a, b)) {
                peak_a[K] = a;
                peak_b[K] = b;
                K++;
            }
        }
    const int32_t Kc = K < capacity ? K : capacity;
    *num_centroids = K;
    for (int32_t k = 0; k < Kc; k++) {
        cpe_oracle_centroid *c = &centroids[k];
        c->bin_x = peak_a[k];
        c->bin_y = peak_b[k];
        c->x = (float)(((double)(peak_a[k] + 1) * (double)W) / (double)(bins_w + 1));
        c->y = (float)(((double)(peak_b[k] + 1) * (double)H) / (double)(bins_h + 1));
        c->score = ldexp((double)Hv[peak_b[k] * bins_w + peak_a[k]], -30);
        c->npix = 0;
        c->reserved = 0;
    }

    /* assignment (Eq7): nearest candidate in the encoded space, d_x + d_y
     * summed exactly (two binary32 values always have an exact binary64
     * sum) */
    for (size_t p = 0; p < npix; p++) {
        labels[p] = 0;
        if (score_map) score_map[p] = 0.0f;
        if (Kc == 0 || !participates(fg, dtype, p, fg_threshold)) continue;
        for (int32_t c = 0; c < twoF; c++) {
            X[c] = to_fixed(load_value(emb, dtype, p * (size_t)D + (size_t)c));
            Y[c] = to_fixed(load_value(emb, dtype, p * (size_t)D + (size_t)(yoff + c)));
        }
        axis_profile(X, Pw, bins_w, twoF, wt, NULL, rx);
        axis_profile(Y, Ph, bins_h, twoF, wt, NULL, ry);
        int32_t best = 0;
        double best_d = (double)rx[peak_a[0]] + (double)ry[peak_b[0]];
        for (int32_t k = 1; k < Kc; k++) {
            double dk = (double)rx[peak_a[k]] + (double)ry[peak_b[k]];
            if (dk < best_d) {
                best_d = dk;
                best = k;
            }
        }
        /* Eq8: the pixel joins mask m only if d(a_m, b_m) < tau */
        if (!(best_d < 4096.0 * tau)) continue;
        labels[p] = best + 1;
        centroids[best].npix += 1;
        if (score_map) score_map[p] = expf(-(float)(best_d * 0x1p-12));
    }

    if (hist) memcpy(hist, Hv, sizeof(uint64_t) * (size_t)nbins);
    if (pal_x) memcpy(pal_x, Pw, sizeof(int16_t) * bins_w * twoF);
    if (pal_y) memcpy(pal_y, Ph, sizeof(int16_t) * bins_h * twoF);
    if (wt_out) memcpy(wt_out, wt, sizeof(uint16_t) * W_KEYS);

    free(Pw); free(Ph); free(wt); free(Hv); free(X); free(Y);
    free(rx); free(ry); free(qx); free(qy); free(peak_a); free(peak_b);
    return CPE_ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* real-valued fp64 decoder: the same steps with no quantisation            */
/* ------------------------------------------------------------------------ */
static void real_palette(int32_t n, int32_t extent, const double *freq, int32_t F, double *pal)
{
    for (int32_t a = 0; a < n; a++) {
        double centre = ((double)(a + 1) * (double)extent) / (double)(n + 1);
        for (int32_t k = 0; k < F; k++) {
            pal[a * 2 * F + 2 * k] = sin(freq[k] * centre);
            pal[a * 2 * F + 2 * k + 1] = cos(freq[k] * centre);
        }
    }
}

static void real_distances(const double *v, const double *pal, int32_t n, int32_t twoF, double *d)
{
    for (int32_t a = 0; a < n; a++) {
        double s = 0.0;
        for (int32_t c = 0; c < twoF; c++) {
            double diff = v[c] - pal[a * twoF + c];
            s += diff * diff;
        }
        d[a] = sqrt(s);
    }
}

int cpe_oracle_decode_real(int32_t H, int32_t W, int32_t D, int32_t dtype,
                           const void *emb, const void *fg,
                           const double *freq_x, const double *freq_y, int32_t n_freq,
                           int32_t bins_w, int32_t bins_h, int32_t capacity,
                           float fg_threshold, double peak_threshold,
                           double *hist, int32_t *peaks, int32_t *num_peaks,
                           int32_t *labels)
{
    if (check_args(H, W, D, dtype, emb, freq_x, freq_y, n_freq, bins_w, bins_h, capacity,
                   fg_threshold, peak_threshold) != CPE_ORACLE_OK || !fg ||
        !hist || !peaks || !num_peaks || !labels)
        return CPE_ORACLE_EINVAL;
    const int32_t F = n_freq, twoF = 2 * n_freq, yoff = D / 2;
    const size_t npix = (size_t)H * (size_t)W;
    const int32_t nbins = bins_w * bins_h;
    double *Pw = malloc(sizeof(double) * bins_w * twoF), *Ph = malloc(sizeof(double) * bins_h * twoF);
    double *vx = malloc(sizeof(double) * twoF), *vy = malloc(sizeof(double) * twoF);
    double *dx = malloc(sizeof(double) * bins_w), *dy = malloc(sizeof(double) * bins_h);
    int32_t *pk = malloc(sizeof(int32_t) * nbins);
    real_palette(bins_w, W, freq_x, F, Pw);
    real_palette(bins_h, H, freq_y, F, Ph);
    for (int32_t i = 0; i < nbins; i++) hist[i] = 0.0;

    for (size_t p = 0; p < npix; p++) {
        if (!(load_value(fg, dtype, p) > fg_threshold)) continue;
        for (int32_t c = 0; c < twoF; c++) {
            vx[c] = (double)load_value(emb, dtype, p * (size_t)D + (size_t)c);
            vy[c] = (double)load_value(emb, dtype, p * (size_t)D + (size_t)(yoff + c));
        }
        real_distances(vx, Pw, bins_w, twoF, dx);
        real_distances(vy, Ph, bins_h, twoF, dy);
        for (int32_t b = 0; b < bins_h; b++)
            for (int32_t a = 0; a < bins_w; a++) hist[b * bins_w + a] += exp(-dx[a]) * exp(-dy[b]);
    }
    int32_t K = 0;
    for (int32_t b = 0; b < bins_h; b++)
        for (int32_t a = 0; a < bins_w; a++)
            if (hist[b * bins_w + a] > peak_threshold && is_peak_f64(hist, bins_w, bins_h, a, b))
                pk[K++] = b * bins_w + a;
    *num_peaks = K;
    const int32_t Kc = K < capacity ? K : capacity;
    for (int32_t k = 0; k < Kc; k++) peaks[k] = pk[k];
    for (size_t p = 0; p < npix; p++) {
        labels[p] = 0;
        if (Kc == 0 || !(load_value(fg, dtype, p) > fg_threshold)) continue;
        for (int32_t c = 0; c < twoF; c++) {
            vx[c] = (double)load_value(emb, dtype, p * (size_t)D + (size_t)c);
            vy[c] = (double)load_value(emb, dtype, p * (size_t)D + (size_t)(yoff + c));
        }
        real_distances(vx, Pw, bins_w, twoF, dx);
        real_distances(vy, Ph, bins_h, twoF, dy);
        int32_t best = 0;
        double best_d = dx[pk[0] % bins_w] + dy[pk[0] / bins_w];
        for (int32_t k = 1; k < Kc; k++) {
            double d = dx[pk[k] % bins_w] + dy[pk[k] / bins_w];
            if (d < best_d) {
                best_d = d;
                best = k;
            }
        }
        labels[p] = best + 1;
    }
    free(Pw); free(Ph); free(vx); free(vy); free(dx); free(dy); free(pk);
    return CPE_ORACLE_OK;
}
