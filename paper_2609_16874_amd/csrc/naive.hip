// naive.hip -- the per-tuple decoder of the prior work the paper measures
// against (Section 3.2, "Histogram Accumulation" and "Mask Aggregation";
// Table 3, "Naive"), as an ablation on this GPU.
//
// Real-valued definition (Section 3.1) in fp32, no quantisation:
//   d_x(p, a) = |x^(p) - P_w(a)|, d_y(p, b) likewise (Eq4, real palettes);
//   H(a, b)   = sum over participating p of e^-d_x e^-d_y (Eq6), one thread
//               per (pixel, bin) tuple, each recomputing both distances and
//               adding its weight with a float atomicAdd into the global
//               histogram: the order of the additions, and so the last bits
//               of H, vary from run to run;
//   peaks     strict 8-neighbour maxima above the threshold (the
//             local-maxima search), listed in bin order by one thread;
//   labels    one thread per (pixel, candidate) tuple recomputes the
//             affinity e^-d_x e^-d_y and keeps the largest per pixel with a
//             64-bit atomicMax on (affinity bits, inverted candidate index),
//             so equal affinities go to the lowest index (Eq7); then one
//             thread per pixel writes its label and counts it.
// Nothing is shared with the matrix-core kernels but the handle's bin
// centres.
#include <hip/hip_runtime.h>

#include <cmath>
#include <new>

#include "cpe_decoder.hpp"

namespace cpe {
namespace {

constexpr int kNaiveThreads = 256;
constexpr int64_t kNaiveMaxBlocks = 1 << 16;

// Real distance of one axis block (2F channels from blk) to a palette row.
template <typename T>
__device__ float naive_axis_dist(const T *__restrict__ blk, const float *__restrict__ pal, int twoF)
{
    float s = 0.0f;
    for (int c = 0; c < twoF; c++) {
        const float d = load_scalar<T>(blk + c) - pal[c];
        s += d * d;
    }
    return sqrtf(s);
}

__global__ void k_naive_clear(float *__restrict__ hf, int nb, unsigned long long *__restrict__ keys, int64_t npix)
{
    const int64_t n = npix > nb ? npix : nb;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        if (i < nb) hf[i] = 0.0f;
        if (i < npix) keys[i] = 0ull;
    }
}

// One (pixel, bin) tuple per thread (grid-stride over all tuples).
template <typename T>
__global__ void k_naive_vote(const T *__restrict__ emb, int32_t dstride, int32_t yoff, const T *__restrict__ fg,
                             int64_t npix, float fg_thr, const float *__restrict__ palx,
                             const float *__restrict__ paly, int twoF, int Bw, int Bh, float *__restrict__ hf)
{
    const int nb = Bw * Bh;
    const int64_t ntup = npix * nb;
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < ntup; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t p = t / nb;
        const int bin = (int)(t - p * nb);
        if (!(load_scalar<T>(fg + p) > fg_thr)) continue;
        const int a = bin % Bw, b = bin / Bw;
        const T *row = emb + p * dstride;
        const float dx = naive_axis_dist(row, palx + (size_t)a * twoF, twoF);
        const float dy = naive_axis_dist(row + yoff, paly + (size_t)b * twoF, twoF);
        atomicAdd(hf + bin, expf(-dx) * expf(-dy));
    }
}

// Every bin tests itself; thread 0 lists the candidates in ascending bin
// order and writes the records (pixel counts reset, added by k_naive_labels).
__global__ void k_naive_peaks(const float *__restrict__ hf, int Bw, int Bh, double thr, int cap,
                              const float *__restrict__ cx, const float *__restrict__ cy,
                              cpe_centroid *__restrict__ cents, int32_t *__restrict__ num,
                              int32_t *__restrict__ peaks, int32_t *__restrict__ kinfo)
{
    extern __shared__ unsigned char flag[];   // [Bw * Bh]
    const int nb = Bw * Bh;
    for (int i = threadIdx.x; i < nb; i += blockDim.x) {
        const int a = i % Bw, b = i / Bw;
        const float v = hf[i];
        bool f = (double)v > thr;
        for (int db = -1; db <= 1; db++)
            for (int da = -1; da <= 1; da++) {
                const int na = a + da, nb_ = b + db;
                if ((da || db) && na >= 0 && na < Bw && nb_ >= 0 && nb_ < Bh) f = f && v > hf[nb_ * Bw + na];
            }
        flag[i] = f ? 1 : 0;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int K = 0;
        for (int i = 0; i < nb; i++) {
            if (!flag[i]) continue;
            if (K < cap) {
                const int a = i % Bw, b = i / Bw;
                cpe_centroid rec;
                rec.bin_x = a;
                rec.bin_y = b;
                rec.x = cx[a];
                rec.y = cy[b];
                rec.score = (double)hf[i];
                rec.npix = 0;
                rec.reserved = 0;
                cents[K] = rec;
                peaks[K] = a | (b << 16);
            }
            K++;
        }
        *num = K;
        kinfo[0] = K < cap ? K : cap;
        kinfo[1] = K;
    }
}

// One (pixel, candidate slot) tuple per thread; slots past min(K, cap) exit.
template <typename T>
__global__ void k_naive_aggregate(const T *__restrict__ emb, int32_t dstride, int32_t yoff, const T *__restrict__ fg,
                                  int64_t npix, float fg_thr, const float *__restrict__ palx,
                                  const float *__restrict__ paly, int twoF, const int32_t *__restrict__ peaks,
                                  const int32_t *__restrict__ kinfo, int cap, unsigned long long *__restrict__ keys)
{
    const int Kc = kinfo[0];
    const int64_t ntup = npix * cap;
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < ntup; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t p = t / cap;
        const int k = (int)(t - p * cap);
        if (k >= Kc || !(load_scalar<T>(fg + p) > fg_thr)) continue;
        const int pk = peaks[k], a = pk & 0xffff, b = pk >> 16;
        const T *row = emb + p * dstride;
        const float dx = naive_axis_dist(row, palx + (size_t)a * twoF, twoF);
        const float dy = naive_axis_dist(row + yoff, paly + (size_t)b * twoF, twoF);
        const float e = expf(-dx) * expf(-dy);
        const unsigned long long key = ((unsigned long long)__float_as_uint(e) << 32) | (0xffffffffu - (uint32_t)k);
        atomicMax(keys + p, key);
    }
}

template <typename T>
__global__ void k_naive_labels(const T *__restrict__ fg, int64_t npix, float fg_thr, const int32_t *__restrict__ kinfo,
                               const unsigned long long *__restrict__ keys, int32_t *__restrict__ labels,
                               cpe_centroid *__restrict__ cents)
{
    const int Kc = kinfo[0];
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < npix; p += (int64_t)gridDim.x * blockDim.x) {
        int lab = 0;
        if (Kc > 0 && load_scalar<T>(fg + p) > fg_thr) {
            const int k = (int)(0xffffffffu - (uint32_t)(keys[p] & 0xffffffffull));
            lab = k + 1;
            atomicAdd(&cents[k].npix, 1);
        }
        labels[p] = lab;
    }
}

int grid_for(int64_t work)
{
    const int64_t b = (work + kNaiveThreads - 1) / kNaiveThreads;
    return (int)(b < 1 ? 1 : (b < kNaiveMaxBlocks ? b : kNaiveMaxBlocks));
}

template <typename T>
cpe_status launch_naive(cpe_decoder *h, hipStream_t stream, const void *emb, const void *fg, float fg_thr,
                        double thr, cpe_centroid *cents, int32_t *num, int32_t *labels, float *hist)
{
    const int Bw = h->bins_w, Bh = h->bins_h, nb = Bw * Bh, twoF = 2 * h->F;
    const int64_t npix = (int64_t)h->H * h->W;
    unsigned char *w = h->naive;
    float *palx = reinterpret_cast<float *>(w);
    float *paly = palx + (size_t)Bw * twoF;
    float *hf_own = paly + (size_t)Bh * twoF;
    int32_t *peaks = reinterpret_cast<int32_t *>(hf_own + nb);
    int32_t *kinfo = peaks + h->cap;
    unsigned long long *keys = reinterpret_cast<unsigned long long *>(
        w + (((size_t)(reinterpret_cast<unsigned char *>(kinfo + 2) - w) + 255) & ~(size_t)255));
    float *hf = hist ? hist : hf_own;
    const T *e = static_cast<const T *>(emb);
    const T *g = static_cast<const T *>(fg);
    const int32_t dstride = h->D, yoff = h->D / 2;
    hipLaunchKernelGGL(k_naive_clear, dim3(grid_for(npix > nb ? npix : nb)), dim3(kNaiveThreads), 0, stream, hf, nb,
                       keys, npix);
    hipLaunchKernelGGL(k_naive_vote<T>, dim3(grid_for(npix * nb)), dim3(kNaiveThreads), 0, stream, e, dstride, yoff, g,
                       npix, fg_thr, (const float *)palx, (const float *)paly, twoF, Bw, Bh, hf);
    hipLaunchKernelGGL(k_naive_peaks, dim3(1), dim3(kNaiveThreads), (size_t)nb, stream, (const float *)hf, Bw, Bh, thr,
                       h->cap, h->tb.cx, h->tb.cy, cents, num, peaks, kinfo);
    hipLaunchKernelGGL(k_naive_aggregate<T>, dim3(grid_for(npix * h->cap)), dim3(kNaiveThreads), 0, stream, e, dstride,
                       yoff, g, npix, fg_thr, (const float *)palx, (const float *)paly, twoF, (const int32_t *)peaks,
                       (const int32_t *)kinfo, h->cap, keys);
    hipLaunchKernelGGL(k_naive_labels<T>, dim3(grid_for(npix)), dim3(kNaiveThreads), 0, stream, g, npix, fg_thr,
                       (const int32_t *)kinfo, (const unsigned long long *)keys, labels, cents);
    return hipGetLastError() == hipSuccess ? CPE_OK : CPE_ERR_HIP;
}

}  // namespace
}  // namespace cpe

using namespace cpe;

extern "C" cpe_status cpe_decode_naive(cpe_decoder *h, hipStream_t stream, const void *emb, const void *fg, int32_t H,
                                       int32_t W, float fg_threshold, double peak_threshold,
                                       cpe_centroid *centroids, int32_t *num_centroids, int32_t *labels, float *hist)
{
    if (!h || !emb || !fg || !centroids || !num_centroids || !labels) return CPE_ERR_INVALID_ARG;
    if (H != h->H || W != h->W) return CPE_ERR_INVALID_ARG;
    const size_t esz = h->dtype == CPE_F32 ? 4 : 2;
    auto aligned = [](const void *p, size_t a) { return ((uintptr_t)p % a) == 0; };
    if (!aligned(emb, esz) || !aligned(fg, esz) || !aligned(labels, 4) || !aligned(centroids, 8) ||
        !aligned(num_centroids, 4) || (hist && !aligned(hist, 4)))
        return CPE_ERR_INVALID_ARG;
    if (!std::isfinite(fg_threshold) || !std::isfinite(peak_threshold)) return CPE_ERR_INVALID_ARG;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return CPE_ERR_HIP;
    if (dev != h->device) return CPE_ERR_INVALID_ARG;
    if (!h->naive) {   // first use: real palettes, own histogram, peak list, per-pixel keys
        const int nb = h->bins_w * h->bins_h, twoF = 2 * h->F;
        const size_t head = ((size_t)(h->bins_w + h->bins_h) * twoF + nb) * 4 + (size_t)h->cap * 4 + 8;
        const size_t bytes = ((head + 255) & ~(size_t)255) + (size_t)h->H * h->W * 8;
        unsigned char *w = nullptr;
        if (hipMalloc(&w, bytes) != hipSuccess) return CPE_ERR_OUT_OF_MEMORY;
        const bool ok =
            hipMemcpy(w, h->palf_x.data(), h->palf_x.size() * 4, hipMemcpyHostToDevice) == hipSuccess &&
            hipMemcpy(w + h->palf_x.size() * 4, h->palf_y.data(), h->palf_y.size() * 4, hipMemcpyHostToDevice) ==
                hipSuccess;
        if (!ok) {
            (void)hipFree(w);
            return CPE_ERR_HIP;
        }
        h->naive = w;
        h->naive_bytes = bytes;
    }
    if (h->dtype == CPE_F32)
        return launch_naive<float>(h, stream, emb, fg, fg_threshold, peak_threshold, centroids, num_centroids, labels,
                                   hist);
    return launch_naive<_Float16>(h, stream, emb, fg, fg_threshold, peak_threshold, centroids, num_centroids, labels,
                                  hist);
}
