// cpe_decode.hip -- gfx950 decoder for sinusoidal centroid encodings: the C
// ABI of include/cpe_decode.h.
//
// Host side: argument checking, construction of the Eq9 palettes and the
// distance-bucket tables in fp64 (once, at create), one device allocation
// for all constants and scratch, and the launch sequence of cpe_decode.
//
// Launches per frame on the caller's stream (launch.hpp), no allocation, no
// host synchronisation, no host copy:
//   compact participating-pixel list, vote histograms cleared (k_compact);
//   vote    per-pixel recovery + soft voting into replicated 64-bit histograms
//           (k_vote_mfma, one pass per block of 32 x 32 bins);
//   peaks   local-maxima search and compaction (k_peaks, grids above 32 x 32);
//   assign  nearest-candidate assignment, label and score write-out, pixel
//           counts (k_assign_mfma, whose workgroups extract the peaks in
//           their prologue, for grids up to 32 x 32; k_assign_generic above).
// cpe_decode_masks expands a label map into binary masks (masks.hip).

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "cpe_decoder.hpp"
#include "k_compact.hpp"

using namespace cpe;

namespace {

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

long long peak_cut(double theta)
{
    const double t = std::floor(theta * 1073741824.0);
    if (t < -1.0) return -1;
    if (t > 4.0e18) return 4000000000000000000LL;
    return (long long)t;
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// List entries a frame of npix pixels may need: the compaction launch's
// slices hold npix entries with at most one slice (slice_pixels) of slack;
// the folded compaction's segments (one per workgroup, each a range of a
// multiple of 8 pixels) at most 8 entries per workgroup, which that slice
// covers.
static_assert(kCompactSpan >= 8 * kMaxSlices, "one compaction slice covers the folded segments' slack");
constexpr int64_t list_entries(int64_t npix)
{
    return npix + slice_pixels(npix);
}

// Eq8 on distance sums D in units of 1/4096: D / 4096 < tau  <=>  D < 4096 tau
// (exact scaling; +inf keeps every pixel, tau <= 0 none).
double tau4096(double tau) { return tau * 4096.0; }

cpe_status decode_frame(cpe_decoder *h, const Scratch *sc, hipStream_t stream, const void *emb, const void *fg,
                        int32_t H, int32_t W, float fg_threshold, double peak_threshold, double tau,
                        cpe_centroid *centroids, int32_t *num_centroids, int32_t *labels, float *score_map)
{
    if (!h || !emb || !centroids || !num_centroids || !labels) return CPE_ERR_INVALID_ARG;
    if (H != h->H || W != h->W) return CPE_ERR_INVALID_ARG;
    const size_t esz = h->dtype == CPE_F32 ? 4 : 2;
    if (!aligned(emb, 16) || (fg && !aligned(fg, esz)) || !aligned(labels, 16) || !aligned(centroids, 8) ||
        !aligned(num_centroids, 4) || (score_map && !aligned(score_map, 4)))
        return CPE_ERR_INVALID_ARG;
    if (!std::isfinite(fg_threshold) || !std::isfinite(peak_threshold)) return CPE_ERR_INVALID_ARG;
    if (std::isnan(tau) || tau == -INFINITY) return CPE_ERR_INVALID_ARG;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return CPE_ERR_HIP;
    if (dev != h->device) return CPE_ERR_INVALID_ARG;
    const FrameArgs fa{stream,       emb,       fg,            fg_threshold, peak_cut(peak_threshold),
                       tau4096(tau), centroids, num_centroids, labels,       score_map};
    const Scratch &s = sc ? *sc : h->sc;
    if (h->dtype == CPE_F32) return h->F <= 8 ? launch_f32_lo(h, s, fa) : launch_f32_hi(h, s, fa);
    return h->F <= 8 ? launch_f16_lo(h, s, fa) : launch_f16_hi(h, s, fa);
}

// Distance at the centre of an m-bit bucket of fl32(S+1) (0 for S = 0).
double centre_distance(int key, int m)
{
    if (key == 0) return 0.0;
    const int e = key >> m, t = key & ((1 << m) - 1);
    return std::sqrt(std::ldexp(1.0 + ((double)t + 0.5) / (double)(1 << m), e) - 1.0) / 4096.0;
}

uint16_t f16_bits(int v)   // exact for the small integers used here (|v| <= 2048)
{
    const _Float16 hv = (_Float16)(float)v;
    uint16_t b;
    std::memcpy(&b, &hv, 2);
    return b;
}

// ---------------------------------------------------------------------------
// Per-frame scratch of cpe_decode_noalloc: a static device array, one copy
// per device, for frames of up to kStaticMaxPixels pixels and any bin grid.
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is looked up once per device (hipGetSymbolAddress, with the
// device current, from cpe_decode_create) and only that address is used.
// ---------------------------------------------------------------------------
constexpr int64_t kStaticMaxPixels = 1LL << 21;     // 2,097,152 pixels, e.g. 1024 x 2048
constexpr int kStaticMaxBins = kMaxBins * kMaxBins;
constexpr size_t kStaticSet = (size_t)kReplicas * kStaticMaxBins;                // words per histogram set
constexpr size_t kStaticHrep = 0;                                               // [2][kReplicas][bins]
constexpr size_t kStaticHlast = kStaticHrep + 2 * kStaticSet * 8;
constexpr size_t kStaticPeaks = kStaticHlast + (size_t)kStaticMaxBins * 8;
constexpr size_t kStaticKinfo = kStaticPeaks + (size_t)kStaticMaxBins * 4;
constexpr size_t kStaticCounts = kStaticKinfo + 256;
constexpr size_t kStaticList = kStaticCounts + (size_t)kMaxSlices * 4;
constexpr size_t kStaticBytes = kStaticList + (size_t)list_entries(kStaticMaxPixels) * 4;
static_assert(kStaticMaxPixels <= (int64_t)kMaxSlices * kCompactSpan, "one compaction step per slice: one slice "
              "of kCompactSpan pixels bounds the list's tail");
static_assert(kStaticMaxPixels <= kFusedMaxPixels, "the folded compaction serves every frame of the static scratch");

__device__ __align__(256) unsigned char scratch[kStaticBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
unsigned char *g_scratch[kMaxDevices];     // device address of `scratch` per device (null: not looked up)
int g_parity[kMaxDevices];                 // histogram set of the next frame in `scratch`, per device
size_t g_dirty[kMaxDevices][2];            // words of each set that may be nonzero, per device

// Look up the device address of `scratch` on the current device `dev` and
// clear its histogram sets, once.
bool init_static_scratch(int dev)
{
    if (dev < 0 || dev >= kMaxDevices) return false;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch[dev]) return true;
    void *ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return false;
    unsigned char *base = static_cast<unsigned char *>(ptr);
    if (hipMemset(base + kStaticHrep, 0, 2 * kStaticSet * 8) != hipSuccess || hipDeviceSynchronize() != hipSuccess)
        return false;
    g_parity[dev] = 0;
    g_dirty[dev][0] = g_dirty[dev][1] = 0;
    g_scratch[dev] = base;
    return true;
}

unsigned char *static_scratch(int dev)
{
    if (dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    return g_scratch[dev];
}

// Its sets have the largest grid's stride, so that handles of any grid
// sharing the array find the set they start on clear.
Scratch static_layout(unsigned char *base, int dev)
{
    Scratch sc;
    sc.hrep = reinterpret_cast<unsigned long long *>(base + kStaticHrep);
    sc.set_stride = kStaticSet;
    sc.parity = &g_parity[dev];
    sc.dirty = g_dirty[dev];
    sc.hlast = reinterpret_cast<unsigned long long *>(base + kStaticHlast);
    sc.peaks = reinterpret_cast<int32_t *>(base + kStaticPeaks);
    sc.kinfo = reinterpret_cast<int32_t *>(base + kStaticKinfo);
    sc.counts = reinterpret_cast<int32_t *>(base + kStaticCounts);
    sc.list = reinterpret_cast<int32_t *>(base + kStaticList);
    return sc;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

const char *cpe_status_string(cpe_status s)
{
    switch (s) {
    case CPE_OK: return "ok";
    case CPE_ERR_INVALID_ARG: return "invalid argument";
    case CPE_ERR_UNSUPPORTED: return "unsupported configuration";
    case CPE_ERR_OUT_OF_MEMORY: return "out of device memory";
    case CPE_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

cpe_status cpe_decode_create(cpe_decoder **out, int32_t H, int32_t W, int32_t D, cpe_dtype dtype,
                             const double *freq_x, const double *freq_y, int32_t n_freq, int32_t bins_w,
                             int32_t bins_h, int32_t centroid_capacity)
{
    if (!out) return CPE_ERR_INVALID_ARG;
    *out = nullptr;
    if (H < 1 || W < 1 || (int64_t)H * W > kMaxPixels) return CPE_ERR_INVALID_ARG;
    if (n_freq < 1 || n_freq > kMaxF || D < 4 * n_freq || D % 2 != 0 || D > 1 << 16) return CPE_ERR_INVALID_ARG;
    if (dtype != CPE_F32 && dtype != CPE_F16) return CPE_ERR_INVALID_ARG;
    // a longer encoding (low harmonics only) is read as two 16-byte aligned blocks
    if (D != 4 * n_freq && (D * (dtype == CPE_F16 ? 2 : 4)) % 32 != 0) return CPE_ERR_UNSUPPORTED;
    if (!freq_x || !freq_y) return CPE_ERR_INVALID_ARG;
    if (bins_w < 1 || bins_w > kMaxBins || bins_h < 1 || bins_h > kMaxBins) return CPE_ERR_INVALID_ARG;
    if (centroid_capacity < 1 || centroid_capacity > bins_w * bins_h) return CPE_ERR_INVALID_ARG;
    for (int k = 0; k < n_freq; k++)
        if (!std::isfinite(freq_x[k]) || !std::isfinite(freq_y[k])) return CPE_ERR_INVALID_ARG;

    cpe_decoder *h = new (std::nothrow) cpe_decoder();
    if (!h) return CPE_ERR_OUT_OF_MEMORY;
    h->H = H;
    h->W = W;
    h->D = D;
    h->F = n_freq;
    h->bins_w = bins_w;
    h->bins_h = bins_h;
    h->cap = centroid_capacity;
    h->dtype = dtype;
    if (hipGetDevice(&h->device) != hipSuccess) {
        delete h;
        return CPE_ERR_HIP;
    }
    // the device address of cpe_decode_noalloc's scratch on this device (a
    // failed lookup only makes that entry point report CPE_ERR_HIP)
    (void)init_static_scratch(h->device);
    const int F = n_freq, twoF = 2 * n_freq, nb = bins_w * bins_h;

    // Eq9 palettes: gamma at the bin centres (a+1) * extent / (n+1), x4096.
    auto palette = [&](int n, int extent, const double *freq, std::vector<int16_t> &pal, std::vector<float> &centres) {
        pal.assign((size_t)n * twoF, 0);
        centres.assign(n, 0.0f);
        for (int a = 0; a < n; a++) {
            const double c = ((double)(a + 1) * (double)extent) / (double)(n + 1);
            centres[a] = (float)c;
            for (int k = 0; k < F; k++) {
                const double ph = freq[k] * c;
                pal[(size_t)a * twoF + 2 * k] = (int16_t)std::rint(4096.0 * std::sin(ph));
                pal[(size_t)a * twoF + 2 * k + 1] = (int16_t)std::rint(4096.0 * std::cos(ph));
            }
        }
    };
    std::vector<float> cx, cy;
    palette(bins_w, W, freq_x, h->pal_x, cx);
    palette(bins_h, H, freq_y, h->pal_y, cy);
    // the same encodings unquantised, in fp32 (the per-tuple ablation)
    auto real_palette = [&](int n, int extent, const double *freq, std::vector<float> &pal) {
        pal.assign((size_t)n * twoF, 0.0f);
        for (int a = 0; a < n; a++) {
            const double c = ((double)(a + 1) * (double)extent) / (double)(n + 1);
            for (int k = 0; k < F; k++) {
                pal[(size_t)a * twoF + 2 * k] = (float)std::sin(freq[k] * c);
                pal[(size_t)a * twoF + 2 * k + 1] = (float)std::cos(freq[k] * c);
            }
        }
    };
    real_palette(bins_w, W, freq_x, h->palf_x);
    real_palette(bins_h, H, freq_y, h->palf_y);

    // weight buckets: 2^15 e^-d, d taken at the centre of the 8-bit bucket
    // of fl32(S+1)
    h->wt.resize(kWKeys);
    for (int k = 0; k < kWKeys; k++) h->wt[k] = (uint16_t)std::rint(32768.0 * std::exp(-centre_distance(k, kWMant)));
    // LDS order of the matrix-core kernels: bucket (e, t) at ((e + 31) & 31) << m | t,
    // so that (float bits >> (23 - m)) & (2^(m+5) - 1) indexes it directly
    std::vector<uint32_t> wt_pk(kWKeys);
    for (int k = 0; k < kWKeys; k++) {
        const int e = k >> kWMant, t = k & ((1 << kWMant) - 1);
        const int q = h->wt[k];
        wt_pk[(((e + 31) & 31) << kWMant) | t] = (uint32_t)f16_bits(q & 255) | ((uint32_t)f16_bits(q >> 8) << 16);
    }

    auto pack = [&](int n, const std::vector<int16_t> &pal, std::vector<int32_t> &pk, std::vector<uint32_t> &n2) {
        pk.assign((size_t)n * F, 0);
        n2.assign(n, 0);
        for (int a = 0; a < n; a++) {
            uint32_t s = 0;
            for (int k = 0; k < F; k++) {
                const int16_t lo = pal[(size_t)a * twoF + 2 * k], hi = pal[(size_t)a * twoF + 2 * k + 1];
                pk[(size_t)a * F + k] = (int32_t)(((uint32_t)(uint16_t)lo) | ((uint32_t)(uint16_t)hi << 16));
                s += (uint32_t)(lo * lo) + (uint32_t)(hi * hi);
            }
            n2[a] = s;
        }
    };
    std::vector<int32_t> pkx, pky;
    std::vector<uint32_t> n2x, n2y;
    pack(bins_w, h->pal_x, pkx, n2x);
    pack(bins_h, h->pal_y, pky, n2y);

    // matrix-core operands: -2P = 128 hi + lo with lo in [-64, 63] (|hi| <= 64),
    // as int8 MFMA operands [axis][block of 32 bins][kind][64 lanes][16 bytes]:
    // lane l holds bin 32 block + (l & 31) and the K slots 16 g .. 16 g + 15
    // (g = l >> 5), whose channels are those the pixel operand of the same half
    // holds (AxisOp in k_mfma.hpp): for 2F > 16 byte b is channel 8 g + b
    // (b < 8) or 16 + 8 g + b - 8, kind 0 = hi, kind 1 = lo; for 2F <= 16 bytes b
    // and 8 + b both belong to channel 8 g + b, kinds (hi, 0), (lo, hi),
    // (0, lo).  Padded bins and channels are 0, and |P|^2 + 1 per bin (1 for
    // padded bins).
    std::vector<int8_t> pop((size_t)2 * kMaxBinBlocks * kPopKinds * 64 * 16, 0);
    std::vector<uint32_t> np1x(kMaxBinBlocks * 32, 1u), np1y(kMaxBinBlocks * 32, 1u);
    for (int ax = 0; ax < 2; ax++) {
        const int n = ax ? bins_h : bins_w;
        const std::vector<int16_t> &pal = ax ? h->pal_y : h->pal_x;
        auto limb = [&](int bin, int c, int which) -> int {     // which 0: hi, 1: lo
            if (bin >= n || c >= twoF) return 0;
            const int m2 = -2 * (int)pal[(size_t)bin * twoF + c];
            const int lo = ((m2 + 64) & 127) - 64;
            return which ? lo : (m2 - lo) / 128;
        };
        for (int blk = 0; blk < kMaxBinBlocks; blk++)
            for (int l = 0; l < 64; l++) {
                const int bin = 32 * blk + (l & 31), g = l >> 5;
                for (int b = 0; b < 16; b++) {
                    int v[kPopKinds];
                    if (twoF > 16) {
                        const int c = b < 8 ? 8 * g + b : 16 + 8 * g + (b - 8);
                        v[0] = limb(bin, c, 0);
                        v[1] = limb(bin, c, 1);
                        v[2] = 0;
                    } else {
                        const int c = 8 * g + (b & 7);
                        v[0] = b < 8 ? limb(bin, c, 0) : 0;
                        v[1] = b < 8 ? limb(bin, c, 1) : limb(bin, c, 0);
                        v[2] = b < 8 ? 0 : limb(bin, c, 1);
                    }
                    for (int k = 0; k < kPopKinds; k++)
                        pop[((((size_t)ax * kMaxBinBlocks + blk) * kPopKinds + k) * 64 + l) * 16 + b] = (int8_t)v[k];
                }
            }
        std::vector<uint32_t> &np1 = ax ? np1y : np1x;
        const std::vector<uint32_t> &n2 = ax ? n2y : n2x;
        for (int bin = 0; bin < n; bin++) np1[bin] = n2[bin] + 1u;
    }

    // one allocation: constants, replicated histograms, last histogram, peak list, counters
    size_t off = 0;
    auto carve = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    const size_t o_px = carve(pkx.size() * 4), o_py = carve(pky.size() * 4);
    const size_t o_nx = carve(n2x.size() * 4), o_ny = carve(n2y.size() * 4);
    const size_t o_wt = carve(kWKeys * 2);
    const size_t o_cx = carve(cx.size() * 4), o_cy = carve(cy.size() * 4);
    const size_t o_npx = carve(np1x.size() * 4), o_npy = carve(np1y.size() * 4);
    const size_t o_pop = carve(pop.size());
    const size_t o_wpk = carve(wt_pk.size() * 4);
    const size_t o_hrep = carve(2 * (size_t)kReplicas * nb * 8);
    const size_t o_hlast = carve((size_t)nb * 8);
    const size_t o_peaks = carve((size_t)centroid_capacity * 4);
    const size_t o_kinfo = carve(16);
    const size_t o_count = carve((size_t)kMaxSlices * 4);
    const size_t o_list = carve((size_t)list_entries((int64_t)H * W) * 4);
    h->dev_bytes = off;
    if (hipMalloc(&h->dev, off) != hipSuccess) {
        delete h;
        return CPE_ERR_OUT_OF_MEMORY;
    }
    unsigned char *d = h->dev;
    auto up = [&](size_t o, const void *src, size_t bytes) {
        return hipMemcpy(d + o, src, bytes, hipMemcpyHostToDevice) == hipSuccess;
    };
    bool ok = up(o_px, pkx.data(), pkx.size() * 4) && up(o_py, pky.data(), pky.size() * 4) &&
              up(o_nx, n2x.data(), n2x.size() * 4) && up(o_ny, n2y.data(), n2y.size() * 4) &&
              up(o_wt, h->wt.data(), kWKeys * 2) &&
              up(o_cx, cx.data(), cx.size() * 4) && up(o_cy, cy.data(), cy.size() * 4) &&
              up(o_npx, np1x.data(), np1x.size() * 4) && up(o_npy, np1y.data(), np1y.size() * 4) &&
              up(o_pop, pop.data(), pop.size()) &&
              up(o_wpk, wt_pk.data(), wt_pk.size() * 4) &&
              hipMemset(d + o_hrep, 0, 2 * (size_t)kReplicas * nb * 8) == hipSuccess &&
              hipMemset(d + o_hlast, 0, (size_t)nb * 8) == hipSuccess &&
              hipMemset(d + o_kinfo, 0, 16) == hipSuccess && hipMemset(d + o_count, 0, (size_t)kMaxSlices * 4) == hipSuccess &&
              hipDeviceSynchronize() == hipSuccess;
    if (!ok) {
        (void)hipFree(h->dev);
        delete h;
        return CPE_ERR_HIP;
    }
    h->tb.pal_x = reinterpret_cast<const int32_t *>(d + o_px);
    h->tb.pal_y = reinterpret_cast<const int32_t *>(d + o_py);
    h->tb.n2_x = reinterpret_cast<const uint32_t *>(d + o_nx);
    h->tb.n2_y = reinterpret_cast<const uint32_t *>(d + o_ny);
    h->tb.wt = reinterpret_cast<const uint16_t *>(d + o_wt);
    h->tb.cx = reinterpret_cast<const float *>(d + o_cx);
    h->tb.cy = reinterpret_cast<const float *>(d + o_cy);
    h->tb.np1_x = reinterpret_cast<const uint32_t *>(d + o_npx);
    h->tb.np1_y = reinterpret_cast<const uint32_t *>(d + o_npy);
    h->tb.pop = reinterpret_cast<const uint32_t *>(d + o_pop);
    h->tb.wt_pk = reinterpret_cast<const uint32_t *>(d + o_wpk);
    h->sc.hrep = reinterpret_cast<unsigned long long *>(d + o_hrep);
    h->sc.set_stride = (size_t)kReplicas * nb;
    h->parity = 0;
    h->sc.parity = &h->parity;
    h->dirty[0] = h->dirty[1] = 0;
    h->sc.dirty = h->dirty;
    h->sc.hlast = reinterpret_cast<unsigned long long *>(d + o_hlast);
    h->sc.peaks = reinterpret_cast<int32_t *>(d + o_peaks);
    h->sc.kinfo = reinterpret_cast<int32_t *>(d + o_kinfo);
    h->sc.counts = reinterpret_cast<int32_t *>(d + o_count);
    h->sc.list = reinterpret_cast<int32_t *>(d + o_list);
    h->fail_at = -1;
    h->search_mode = 0;
    *out = h;
    return CPE_OK;
}

cpe_status cpe_decode(cpe_decoder *h, hipStream_t stream, const void *emb, const void *fg, int32_t H, int32_t W,
                      float fg_threshold, double peak_threshold, cpe_centroid *centroids, int32_t *num_centroids,
                      int32_t *labels, float *score_map)
{
    if (!fg) return CPE_ERR_INVALID_ARG;
    return decode_frame(h, nullptr, stream, emb, fg, H, W, fg_threshold, peak_threshold, INFINITY, centroids,
                        num_centroids, labels, score_map);
}

cpe_status cpe_decode_ex(cpe_decoder *h, hipStream_t stream, const void *emb, const void *fg, int32_t H, int32_t W,
                         const cpe_decode_options *opt, cpe_centroid *centroids, int32_t *num_centroids,
                         int32_t *labels, float *score_map)
{
    if (!opt || opt->reserved != 0) return CPE_ERR_INVALID_ARG;
    // without a foreground channel the threshold is never read
    const float fg_thr = fg ? opt->fg_threshold : 0.0f;
    return decode_frame(h, nullptr, stream, emb, fg, H, W, fg_thr, opt->peak_threshold, opt->tau, centroids,
                        num_centroids, labels, score_map);
}

cpe_status cpe_decode_noalloc(cpe_decoder *h, hipStream_t stream, const void *emb, const void *fg, int32_t H,
                              int32_t W, const cpe_decode_options *opt, cpe_centroid *centroids,
                              int32_t *num_centroids, int32_t *labels, float *score_map)
{
    if (!h || !opt || opt->reserved != 0) return CPE_ERR_INVALID_ARG;
    if ((int64_t)h->H * h->W > kStaticMaxPixels) return CPE_ERR_UNSUPPORTED;
    unsigned char *base = static_scratch(h->device);
    if (!base) return CPE_ERR_HIP;
    const Scratch sc = static_layout(base, h->device);
    const float fg_thr = fg ? opt->fg_threshold : 0.0f;
    return decode_frame(h, &sc, stream, emb, fg, H, W, fg_thr, opt->peak_threshold, opt->tau, centroids,
                        num_centroids, labels, score_map);
}

cpe_status cpe_decode_masks(cpe_decoder *h, hipStream_t stream, const int32_t *labels, int32_t H, int32_t W,
                            int32_t first, int32_t count, uint8_t *masks)
{
    if (!h || !labels || !masks || !aligned(labels, 16) || !aligned(masks, 16)) return CPE_ERR_INVALID_ARG;
    if (H != h->H || W != h->W) return CPE_ERR_INVALID_ARG;
    if (first < 0 || count < 1 || (int64_t)first + count > h->cap) return CPE_ERR_INVALID_ARG;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return CPE_ERR_HIP;
    if (dev != h->device) return CPE_ERR_INVALID_ARG;
    return launch_masks(stream, labels, (int64_t)H * W, first, count, masks);
}

cpe_status cpe_decode_destroy(cpe_decoder *h)
{
    if (!h) return CPE_OK;
    hipError_t e = hipFree(h->dev);
    if (h->naive && hipFree(h->naive) != hipSuccess) e = hipErrorUnknown;
    delete h;
    return e == hipSuccess ? CPE_OK : CPE_ERR_HIP;
}

cpe_status cpe_decode_get_tables(const cpe_decoder *h, int16_t *pal_x, int16_t *pal_y, uint16_t *weights)
{
    if (!h) return CPE_ERR_INVALID_ARG;
    if (pal_x) std::memcpy(pal_x, h->pal_x.data(), h->pal_x.size() * sizeof(int16_t));
    if (pal_y) std::memcpy(pal_y, h->pal_y.data(), h->pal_y.size() * sizeof(int16_t));
    if (weights) std::memcpy(weights, h->wt.data(), h->wt.size() * sizeof(uint16_t));
    return CPE_OK;
}

cpe_status cpe_decode_get_histogram(cpe_decoder *h, hipStream_t stream, uint64_t *hist)
{
    if (!h || !hist || !aligned(hist, 8)) return CPE_ERR_INVALID_ARG;
    const size_t bytes = (size_t)h->bins_w * h->bins_h * 8;
    return hipMemcpyAsync(hist, h->sc.hlast, bytes, hipMemcpyDeviceToDevice, stream) == hipSuccess ? CPE_OK : CPE_ERR_HIP;
}

cpe_status cpe_decode_test_fail_launch(cpe_decoder *h, int32_t launch)
{
    if (!h || launch < -1 || launch > 2) return CPE_ERR_INVALID_ARG;
    h->fail_at = launch;
    return CPE_OK;
}

cpe_status cpe_decode_test_search_mode(cpe_decoder *h, int32_t mode)
{
    if (!h || mode < 0 || mode > 2) return CPE_ERR_INVALID_ARG;
    h->search_mode = mode;
    return CPE_OK;
}

size_t cpe_decode_workspace_bytes(const cpe_decoder *h) { return h ? h->dev_bytes : 0; }

int32_t cpe_decode_launch_count(const cpe_decoder *h)
{
    if (!h) return 0;
    const bool mfma = h->bins_w <= kMfmaBins && h->bins_h <= kMfmaBins;
    return mfma && fused_plan((int64_t)h->H * h->W).ok ? 2 : 3;
}

cpe_status cpe_decode_set_stage_events(cpe_decoder *h, hipEvent_t *events, int32_t n_events)
{
    if (!h) return CPE_ERR_INVALID_ARG;
    if (!events) {
        h->stage_on = false;
        return CPE_OK;
    }
    if (n_events != CPE_STAGE_EVENTS) return CPE_ERR_INVALID_ARG;
    for (int i = 0; i < CPE_STAGE_EVENTS; i++) {
        if (!events[i]) return CPE_ERR_INVALID_ARG;
        h->stage_ev[i] = events[i];
    }
    h->stage_on = true;
    return CPE_OK;
}

}  // extern "C"
