/*
 * cpe_oracle.c -- plain CPU oracle of the centroid-encoding decoder.
 *
 * TEST INFRASTRUCTURE ONLY (see cpe_oracle.h).  Single-threaded, no SIMD, no
 * blocking, no reordering beyond what each step's definition states.  Built
 * with gcc -O2 and without -ffast-math so that rintf/sqrtf/(float) casts are
 * the IEEE round-to-nearest-even operations the canonical arithmetic names.
 *
 * The steps follow Section 3 of the paper in its own order:
 *   palettes (Eq9)                     -> build_palette()
 *   per-axis distances, weights        -> axis_profile()      (Eq4, Eq5, Eq10)
 *   vote histogram                     -> accumulate over S   (Eq6, Eq11)
 *   local-maxima search                -> is_peak()           (LMS paragraph)
 *   assignment and counts              -> assign()            (Eq7, mask
 *                                                              aggregation)
 *
 * Canonical arithmetic (the reading adopted where the paper fixes no
 * precision; every constant below is part of that contract):
 *   bin centres   x_a = (a+1) W / (B_w+1), y_b = (b+1) H / (B_h+1)  (fp64;
 *                 Eq9 with u = 2x/W - 1 and continuous pixel coordinates)
 *   palette       P[a][2k] = rint(4096 sin(w_k x_a)), P[a][2k+1] =
 *                 rint(4096 cos(w_k x_a)), fp64, stored as int16
 *   LUT           LUT[i] = rint(32768 exp(-i/256)), i = 0..2840, uint16
 *   input         X = clamp(rintf(4096.0f * v), -6144, 6144); NaN -> 0
 *   participation p in S  <=>  (float)fg(p) > fg_threshold
 *   distance      S_x = sum_c (X_c - P[a][c])^2 (exact integer),
 *                 r_x = sqrtf((float)S_x), d_x = r_x / 4096
 *   weight        q_x = LUT[min(rint(r_x * 0.0625f), 2840)]  ~ 2^15 e^-d_x
 *   votes         H[b][a] = sum_{p in S} q_x(p,a) q_y(p,b)    (exact uint64)
 *   peaks         H[b][a] > floor(theta_peak 2^30) and > every in-range
 *                 8-neighbour; listed in ascending b*B_w + a
 *   assignment    D_k = fl32(r_x(a_k) + r_y(b_k)); the smallest k with the
 *                 minimal D_k wins; label = k+1, background 0
 *
 * Pins (tests/test_oracle_*.py), each independent of this file's code:
 *   - LUT closed-form values and monotonicity; palette sin^2+cos^2 = 1;
 *   - the vote histogram against the paper's matrix form E_x^T E_y in fp64
 *     (numpy), within the quantisation error bound;
 *   - brute force on tiny frames: exhaustive scan of every grid position for
 *     the peaks and every candidate for each pixel's assignment;
 *   - noise-free frames whose centroids sit on bin centres decode to the
 *     generating centroids and the generating label map;
 *   - invariants: labels partition the foreground, counts sum to |S|,
 *     peaks pairwise non-adjacent, instance-order independence.
 * The whole pipeline against the paper's own decoder: parity unpinned (no
 * implementation or worked example is published).
 */
#include "cpe_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define FIX_SCALE 4096.0f       /* input and palette fixed-point scale   */
#define X_CLAMP 6144            /* |X| <= 1.5 * 4096                      */
#define LUT_LEN 2841            /* indices 0..2840 (rint(256 d))          */
#define LUT_LAST 2840

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

/* Input to fixed point. */
static int32_t to_fixed(float v)
{
    if (isnan(v)) return 0;
    float t = rintf(FIX_SCALE * v);
    if (t < (float)-X_CLAMP) return -X_CLAMP;
    if (t > (float)X_CLAMP) return X_CLAMP;
    return (int32_t)t;
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

static void build_lut(uint16_t *lut)
{
    for (int32_t i = 0; i < LUT_LEN; i++) lut[i] = (uint16_t)rint(32768.0 * exp(-(double)i / 256.0));
}

/* Eq4/Eq10 for one axis of one pixel: r[a] = sqrtf(S(a)), q[a] = weight. */
static void axis_profile(const int32_t *X, const int16_t *pal, int32_t n, int32_t twoF,
                         const uint16_t *lut, float *r, uint32_t *q)
{
    for (int32_t a = 0; a < n; a++) {
        uint64_t s = 0;
        for (int32_t c = 0; c < twoF; c++) {
            int64_t diff = (int64_t)X[c] - (int64_t)pal[a * twoF + c];
            s += (uint64_t)(diff * diff);
        }
        float ra = sqrtf((float)(uint32_t)s);
        r[a] = ra;
        if (q) {
            int32_t idx = (int32_t)rintf(ra * 0.0625f);
            if (idx > LUT_LAST) idx = LUT_LAST;
            q[a] = lut[idx];
        }
    }
}

static int64_t peak_cut(double theta)
{
    double t = floor(theta * 1073741824.0);
    if (t < -1.0) return -1;
    if (t > 4.0e18) return (int64_t)4000000000000000000LL;
    return (int64_t)t;
}

static int check_args(int32_t H, int32_t W, int32_t D, int32_t dtype, const void *emb, const void *fg,
                      const double *fx, const double *fy, int32_t n_freq, int32_t bw, int32_t bh,
                      int32_t cap, float fg_thr, double peak_thr)
{
    if (H < 1 || W < 1 || (int64_t)H * (int64_t)W > 2147483647LL) return CPE_ORACLE_EINVAL;
    if (n_freq < 1 || n_freq > 16 || D != 4 * n_freq) return CPE_ORACLE_EINVAL;
    if (dtype != 0 && dtype != 1) return CPE_ORACLE_EINVAL;
    if (!emb || !fg || !fx || !fy) return CPE_ORACLE_EINVAL;
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

int cpe_oracle_decode(int32_t H, int32_t W, int32_t D, int32_t dtype,
                      const void *emb, const void *fg,
                      const double *freq_x, const double *freq_y, int32_t n_freq,
                      int32_t bins_w, int32_t bins_h, int32_t capacity,
                      float fg_threshold, double peak_threshold,
                      cpe_oracle_centroid *centroids, int32_t *num_centroids,
                      int32_t *labels, float *score_map,
                      uint64_t *hist, int16_t *pal_x, int16_t *pal_y, uint16_t *lut_out)
{
    if (check_args(H, W, D, dtype, emb, fg, freq_x, freq_y, n_freq, bins_w, bins_h, capacity,
                   fg_threshold, peak_threshold) != CPE_ORACLE_OK ||
        !centroids || !num_centroids || !labels)
        return CPE_ORACLE_EINVAL;

    const int32_t F = n_freq, twoF = 2 * n_freq;
    const size_t npix = (size_t)H * (size_t)W;
    const int32_t nbins = bins_w * bins_h;

    int16_t *Pw = malloc(sizeof(int16_t) * bins_w * twoF);
    int16_t *Ph = malloc(sizeof(int16_t) * bins_h * twoF);
    uint16_t lut[LUT_LEN];
    uint64_t *Hv = calloc((size_t)nbins, sizeof(uint64_t));
    int32_t *X = malloc(sizeof(int32_t) * twoF);
    int32_t *Y = malloc(sizeof(int32_t) * twoF);
    float *rx = malloc(sizeof(float) * bins_w), *ry = malloc(sizeof(float) * bins_h);
    uint32_t *qx = malloc(sizeof(uint32_t) * bins_w), *qy = malloc(sizeof(uint32_t) * bins_h);
    int32_t *peak_a = malloc(sizeof(int32_t) * nbins), *peak_b = malloc(sizeof(int32_t) * nbins);

    /* palettes, preloaded once (Section 3.2, Eq9) and the weight table */
    build_palette(bins_w, W, freq_x, F, Pw);
    build_palette(bins_h, H, freq_y, F, Ph);
    build_lut(lut);

    /* histogram accumulation: H(a,b) = sum_{p in S} E_x(p,a) E_y(p,b) */
    for (size_t p = 0; p < npix; p++) {
        if (!(load_value(fg, dtype, p) > fg_threshold)) continue;
        for (int32_t c = 0; c < twoF; c++) {
            X[c] = to_fixed(load_value(emb, dtype, p * (size_t)D + (size_t)c));
            Y[c] = to_fixed(load_value(emb, dtype, p * (size_t)D + (size_t)(twoF + c)));
        }
        axis_profile(X, Pw, bins_w, twoF, lut, rx, qx);
        axis_profile(Y, Ph, bins_h, twoF, lut, ry, qy);
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

    /* assignment (Eq7): nearest candidate in the encoded space */
    for (size_t p = 0; p < npix; p++) {
        labels[p] = 0;
        if (score_map) score_map[p] = 0.0f;
        if (Kc == 0 || !(load_value(fg, dtype, p) > fg_threshold)) continue;
        for (int32_t c = 0; c < twoF; c++) {
            X[c] = to_fixed(load_value(emb, dtype, p * (size_t)D + (size_t)c));
            Y[c] = to_fixed(load_value(emb, dtype, p * (size_t)D + (size_t)(twoF + c)));
        }
        axis_profile(X, Pw, bins_w, twoF, lut, rx, NULL);
        axis_profile(Y, Ph, bins_h, twoF, lut, ry, NULL);
        int32_t best = 0;
        float best_d = rx[peak_a[0]] + ry[peak_b[0]];
        for (int32_t k = 1; k < Kc; k++) {
            float dk = rx[peak_a[k]] + ry[peak_b[k]];
            if (dk < best_d) {
                best_d = dk;
                best = k;
            }
        }
        labels[p] = best + 1;
        centroids[best].npix += 1;
        if (score_map) score_map[p] = expf(-(best_d * 0x1p-12f));
    }

    if (hist) memcpy(hist, Hv, sizeof(uint64_t) * (size_t)nbins);
    if (pal_x) memcpy(pal_x, Pw, sizeof(int16_t) * bins_w * twoF);
    if (pal_y) memcpy(pal_y, Ph, sizeof(int16_t) * bins_h * twoF);
    if (lut_out) memcpy(lut_out, lut, sizeof(lut));

    free(Pw); free(Ph); free(Hv); free(X); free(Y);
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
    if (check_args(H, W, D, dtype, emb, fg, freq_x, freq_y, n_freq, bins_w, bins_h, capacity,
                   fg_threshold, peak_threshold) != CPE_ORACLE_OK ||
        !hist || !peaks || !num_peaks || !labels)
        return CPE_ORACLE_EINVAL;
    const int32_t F = n_freq, twoF = 2 * n_freq;
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
            vy[c] = (double)load_value(emb, dtype, p * (size_t)D + (size_t)(twoF + c));
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
            vy[c] = (double)load_value(emb, dtype, p * (size_t)D + (size_t)(twoF + c));
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
